// Multi-head latent attention (MLA) decode for gfx950 (MI355X).
//
// One new token per batch element: every query head h attends to all Skv
// positions of the latent cache of its latent head hk = h / (H / Hkv),
//   s_t = scale * (q[h] . kv[t] + q_pe[h] . k_pe[t]),
//   O[h] = sum_t softmax(s)_t kv[t],   LSE[h] = ln sum_t exp(s_t),
// the computation of the paper's appendix listing "Implementation of
// FlashMLA with TileLang" (scores from the latent and the rotary parts
// accumulated into one tile, online softmax over cache tiles, the latent
// cache serving again as the value).  The design is this library's own for
// CDNA4:
//
//  * One workgroup of four wave64s (one per SIMD) owns HB = 64 query heads
//    of one latent head of one batch element, and one range of cache tiles
//    (a key split).  The waves form two pairs, each pair owning 32 heads.
//    S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (A = 32 cache rows from LDS,
//    B = the query of the pair's heads, held in registers for the whole
//    kernel): the two waves of a pair each take half of the 576-wide
//    contraction (18 of its 36 k-steps) and exchange their partial scores
//    through LDS, so both hold the full scores of the tile.  In the
//    accumulator layout lane l owns head l % 32, so the softmax row
//    reductions are in-lane plus one v_permlane32_swap.
//  * O^T += V^T P^T: the bf16 weights already sit in the B-operand layout;
//    V^T comes from the same latent rows in LDS through the transpose read
//    ds_read_b64_tr_b16.  Each wave of a pair accumulates half (256) of the
//    512 output dims of its 32 heads: 128 fp32 registers per lane, kept in
//    the matrix-core registers; LDS holds only the streamed cache tiles and
//    the score exchange.
//  * Cache tiles of 32 positions go global -> LDS by DMA (buffer_load_dwordx4
//    ... lds) into a ring of four buffers, three tiles ahead of the one in
//    use: the latent part [32][512] and the rotary part [32][64] in two
//    regions.  16-byte chunks are XOR-swizzled so that the
//    score operand reads (ds_read_b128) and the transpose reads of the same
//    latent rows are both bank-conflict free (chunk c of latent row r at
//    c ^ (((r & 3) << 2) | ((r >> 2) & 3)), of rotary row r at c ^ ((r >> 1) & 7)).
//  * Online softmax as in the attention kernel: the running max m is raised
//    when a head's tile max passes m + min(8, max(0, log2(l / 4))) (l the
//    lane's running sum), so a position that could dominate a head is
//    weighted exactly 1; weights rounded to bf16 for the P V product, fp32
//    sums.
//  * Key splits write per-split (O_s, LSE_s) to a workspace; the merge kernel
//    of split_combine.h combines them exactly.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tileattn.h"
#include "split_combine.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int DL = 512;              // latent width (query, cache, output)
constexpr int DR = 64;               // rotary width (query, key)
constexpr int BN = 32;               // cache positions per tile
constexpr int NT = 256;              // threads per workgroup (4 waves)
constexpr int HB = 64;               // query heads per workgroup (two wave pairs x 32)
constexpr int KKL = DL / 16;         // MFMA k-steps over the latent part
constexpr int KKR = DR / 16;         // ... over the rotary part
constexpr int KKH = (KKL + KKR) / 2; // k-steps per wave of a pair
constexpr int DH = DL / 2;           // output dims per wave
constexpr int DBV = DH / 32;         // 32-row blocks of the wave's O^T
constexpr int LAT_BYTES = BN * DL * 2;
constexpr int ROT_BYTES = BN * DR * 2;
constexpr int LAT_PER_THREAD = BN * (DL / 8) / NT;   // 16-byte DMA chunks per thread
constexpr int ROT_PER_THREAD = BN * (DR / 8) / NT;
constexpr int NXCD = 8;
constexpr float LOG2E = 1.44269504088896340736f;
constexpr float LN2 = 0.69314718055994530942f;
constexpr float RESCALE_SLACK = 8.0f;       // base-2 headroom: weights never exceed 2^8
constexpr float RAISE_SHARE_LOG2 = -2.0f;   // log2 of the share (1/4) of l a position may
                                            // weigh before the max is raised
[[maybe_unused]] constexpr int BUF_RSRC_WORD3 = 0x00020000;
static_assert(LAT_PER_THREAD == 8 && ROT_PER_THREAD == 1, "tile/thread mismatch");

struct MArgs {
    const uint16_t *Q, *Qpe, *KV, *Kpe;
    float *O, *LSE;           // output, or split 0 of the partial results
    size_t o_split, l_split;  // element strides between splits
    int B, H, Hkv, Skv;
    int g;                    // H / Hkv query heads per latent head
    int n_hblk;               // workgroups over the heads of one latent head
    int n_split, split_tiles;
    int n_wg;
    float c;                  // scale * log2(e)
};

// 16-byte chunk swizzles (XOR within aligned groups of 16, resp. 8, chunks)
__device__ __forceinline__ int lat_swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int rot_swz(int r) { return (r >> 1) & 7; }

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float max_halves(float x)
{
    const u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                     false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float sum_halves(float x)
{
    const u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                     false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Tile DMA is issued as inline assembly (buffer_load_dwordx4 ... lds), so
// the compiler does not track it: it then never drains the tile loads in
// flight before an LDS read (it cannot tell which buffer a DMA writes), and
// the kernel waits for them itself with these vmcnt waits.  The kernel's
// only other vector-memory operations are the query loads before the first
// DMA and the output stores after the last wait.
constexpr int DMA_PER_TILE = LAT_PER_THREAD + ROT_PER_THREAD;   // per thread
static_assert(DMA_PER_TILE == 9, "vmcnt encodings below");
// s_waitcnt vmcnt(n) (low 4 bits of n in [3:0], high 2 bits in [15:14]),
// expcnt and lgkmcnt left at their maxima
__device__ __forceinline__ void wait_dma_tiles_left(int tiles)   // tiles: 0, 1 or 2, uniform
{
    if (tiles >= 2)
        __builtin_amdgcn_s_waitcnt(0x4F72);   // vmcnt(18)
    else if (tiles == 1)
        __builtin_amdgcn_s_waitcnt(0x0F79);   // vmcnt(9)
    else
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
}

typedef uint32_t u32x4s __attribute__((ext_vector_type(4)));

// A raw buffer resource (stride 0, 32-bit format, range-checked) in scalar
// registers.
__device__ __forceinline__ u32x4s buffer_rsrc(const void *base, uint32_t bytes)
{
    const uint64_t a = (uint64_t)(uintptr_t)base;
    return u32x4s{(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a),
                  (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xFFFFu),
                  (uint32_t)__builtin_amdgcn_readfirstlane(bytes), (uint32_t)BUF_RSRC_WORD3};
}

// One 16-byte-per-lane DMA: lane l's 16 bytes at byte `voff` of the buffer
// land at LDS address `lds` + 16 l (`lds` wave-uniform).
// M0 is an operand of the statement, so the compiler sets it (and keeps any
// value of its own) around the load.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, u32x4s rsrc)
{
    asm volatile("s_nop 0\n\t"   // one wait state between the M0 write and the load
                 "buffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voff), "s"(rsrc), "{m0}"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}

// LDS exchange between the two waves of a pair: each wave's partial scores
// (its half of the 576-wide dot products) in the accumulator layout, and at
// the end nothing else (both waves then hold identical softmax state)
struct Xchg {
    float4 s[4][4][64];   // [wave][r / 4][lane]: 16-byte accesses, lanes contiguous
};

struct Mla {
    const MArgs &a;
    int wave, lane, col, half;
    int k_half;                     // which 18 of the 36 score k-steps this wave computes
    int dim_half;                   // which 256 output dims this wave accumulates
    const uint16_t *kv_b, *kpe_b;   // cache of (batch, latent head) at position 0
    uint32_t lat_off[4], rot_off;   // per-lane DMA source offsets (see init_dma)
    bf16x8 qreg[KKH];               // the query's k-steps 18 k_half .. +18
    f32x16 acc_o[DBV];
    float m_run, l_run;
    float m_trig;   // the running max is raised when a tile max exceeds this

    __device__ Mla(const MArgs &args) : a(args) {}

    // Latent DMA slot i*NT + 64w + l (i < 8) is row r = 4i + w, stored chunk
    // sc = l, fetched from source chunk sc ^ lat_swz(r) = l ^ (w << 2) ^ (i & 3):
    // four per-lane offsets (i & 3), plus 4(i & ~3) rows of pitch.  Rotary
    // slot 64w + l is row 8w + l / 8, chunk l % 8, fetched from chunk
    // (l % 8) ^ rot_swz(row).
    __device__ __forceinline__ void init_dma()
    {
        const int wave_u = __builtin_amdgcn_readfirstlane(wave);
        const uint32_t lat_pitch = (uint32_t)a.Hkv * DL * 2, rot_pitch = (uint32_t)a.Hkv * DR * 2;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            lat_off[i] = (4 * i + wave_u) * lat_pitch + 16 * (lane ^ (wave_u << 2) ^ i);
        const int r = 8 * wave_u + lane / 8;
        rot_off = r * rot_pitch + 16 * ((lane % 8) ^ rot_swz(r));
    }

    // DMA cache tile j (positions j*BN ..) into the latent and rotary
    // buffers.  Each buffer resource starts at the tile and ends after its
    // last valid row; a row past Skv re-reads the last valid row (its scores
    // are masked), so no lane addresses outside the cache.
    __device__ __forceinline__ void dma_tile(int j, unsigned char *lat, unsigned char *rot) const
    {
        const int valid = min(BN, a.Skv - j * BN);
        const size_t row0 = (size_t)j * BN * a.Hkv;
        const uint32_t lat_pitch = (uint32_t)a.Hkv * DL * 2, rot_pitch = (uint32_t)a.Hkv * DR * 2;
        const u32x4s rl = buffer_rsrc(kv_b + row0 * DL, (valid - 1) * lat_pitch + DL * 2);
        const u32x4s rr = buffer_rsrc(kpe_b + row0 * DR, (valid - 1) * rot_pitch + DR * 2);
        const int wave_u = __builtin_amdgcn_readfirstlane(wave);
        const int last = valid - 1;
        const uint32_t lat_base = lds_addr(lat), rot_base = lds_addr(rot);
#pragma unroll
        for (int i = 0; i < LAT_PER_THREAD; ++i) {
            // row 4i + w, or the last valid row past it; lat_off[i & 3] holds
            // row 4(i & 3) + w.  (The difference can be negative: it is added
            // to the vector offset modulo 2^32.)
            const int row = 4 * i + wave_u;
            const int src = row > last ? last : row;
            const uint32_t o =
                lat_off[i & 3] + (uint32_t)((src - 4 * (i & 3) - wave_u) * (int)lat_pitch);
            dma16(lat_base + (i * NT + wave_u * 64) * 16, o, rl);
        }
        {
            // row 8w + l/8 is lane-dependent: clamp per lane
            const int row = 8 * wave_u + lane / 8;
            const int shift = row > last ? row - last : 0;
            dma16(rot_base + wave_u * 64 * 16, rot_off - (uint32_t)shift * rot_pitch, rr);
        }
    }

    // Partial S^T[position][head] over this wave's 18 k-steps (288 of the
    // 576 key dims) for the tile's 32 positions; k-step kk < 32 is latent
    // chunk 2kk + half, kk >= 32 rotary chunk 2(kk - 32) + half.  Two
    // interleaved accumulation chains.
    template <int KH>
    __device__ __forceinline__ void scores(const unsigned char *lat, const unsigned char *rot,
                                           f32x16 &s) const
    {
        f32x16 s0, s1;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            s0[r] = 0.f;
            s1[r] = 0.f;
        }
        const int row = col;
#pragma unroll
        for (int i = 0; i < KKH; ++i) {
            const int kk = KH * KKH + i;
            bf16x8 av;
            if (kk < KKL)   // byte 256 (kk >> 3) + 16 ((2 (kk & 7) + half) ^ lat_swz(row))
                av = *(const bf16x8 *)(lat + row * (DL * 2) + 256 * (kk >> 3) +
                                       16 * ((2 * (kk & 7) + half) ^ lat_swz(row)));
            else
                av = *(const bf16x8 *)(rot + row * (DR * 2) +
                                       16 * ((2 * (kk - KKL) + half) ^ rot_swz(row)));
            if (i & 1)
                s1 = mfma32(av, qreg[i], s1);
            else
                s0 = mfma32(av, qreg[i], s0);
            if ((i & 7) == 7)   // bound how far ahead operand reads are issued
                __builtin_amdgcn_sched_barrier(0);
        }
        s = s0 + s1;
    }

    // O^T += V^T P^T for one tile: the weights pk (B-operand layout) of its
    // 32 positions and the transpose reads of its latent rows for this
    // wave's 256 output dims
    __device__ __forceinline__ void pv(const uint32_t (&pk)[8], const unsigned char *lat)
    {
        // MFMA k-slot t of half h stands for position 16ks + 4h + t (t < 4)
        // or 16ks + 8 + 4h + t-4, matching where the accumulator left P
        const int gq = lane >> 4, sl = lane & 15;
        const int c = 2 * (gq & 1) + ((sl & 3) >> 1);
        const int byte_in = 8 * (sl & 1);
#pragma unroll
        for (int ks = 0; ks < BN / 16; ++ks) {
            const u32x4 bw = {pk[4 * ks], pk[4 * ks + 1], pk[4 * ks + 2], pk[4 * ks + 3]};
            const bf16x8 bv = __builtin_bit_cast(bf16x8, bw);
            const int row0 = 16 * ks + 4 * half + (sl >> 2);
            const int row1 = row0 + 8;
            // dims d = 256 dim_half + 32db + 16(gq & 1) + 4(sl & 3): chunk
            // d >> 3 = 32 dim_half + 4db + c, XOR-swizzled within its group of
            // 16: byte 512 dim_half + 256 (db >> 2) + 16 ((4(db & 3) + c) ^ f)
            const unsigned char *r0 = lat + row0 * (DL * 2) + 512 * dim_half + byte_in;
            const unsigned char *r1 = lat + row1 * (DL * 2) + 512 * dim_half + byte_in;
            const int f0 = lat_swz(row0), f1 = lat_swz(row1);
#pragma unroll
            for (int db = 0; db < DBV; ++db) {
                const unsigned char *p0 = r0 + 256 * (db >> 2) + 16 * ((4 * (db & 3) + c) ^ f0);
                const unsigned char *p1 = r1 + 256 * (db >> 2) + 16 * ((4 * (db & 3) + c) ^ f1);
                const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p0);
                const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p1);
                const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
                const u32x4 aw = {l2[0], l2[1], h2[0], h2[1]};
                acc_o[db] = mfma32(__builtin_bit_cast(bf16x8, aw), bv, acc_o[db]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // One cache tile j, software-pipelined one tile deep: the partial
    // scores of tile j, then the P V of tile j-1 (its weights pk from the
    // previous step, its rows still in the previous buffer) while the
    // partial scores travel to the partner wave; after the barrier, tile
    // j+3 goes into that previous buffer, and the softmax of tile j leaves
    // its weights in pk for the next step.  KH = k_half, a template argument
    // so that the query's k-steps are indexed statically.
    template <bool MASKED, int KH, bool PREV>
    __device__ __forceinline__ void step(int j, int j_hi, const unsigned char *lat,
                                         const unsigned char *rot, unsigned char *lat_p,
                                         unsigned char *rot_p, uint32_t (&pk)[8], Xchg &x)
    {
        f32x16 s;
        scores<KH>(lat, rot, s);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
            x.s[wave][r4][lane] = float4{s[4 * r4], s[4 * r4 + 1], s[4 * r4 + 2], s[4 * r4 + 3]};
        if (PREV)
            pv(pk, lat_p);
        __syncthreads();
        // every wave is past tile j-1 now: its buffers take tile j+3
        if (j + 3 < j_hi)
            dma_tile(j + 3, lat_p, rot_p);
        // (k-half 0) + (k-half 1) in the same order on both waves, so that
        // the pair computes bitwise the same scores
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            const float4 o = x.s[wave ^ 1][r4][lane];
            const float ov[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 4 * r4 + e;
                s[r] = KH == 0 ? s[r] + ov[e] : ov[e] + s[r];
            }
        }

        // lane holds positions j*BN + 8(r/4) + 4half + r%4 of head col
        float mx = -INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            if (MASKED) {
                const int pos = j * BN + 8 * (r >> 2) + 4 * half + (r & 3);
                s[r] = pos < a.Skv ? s[r] : -INFINITY;
            }
            mx = fmaxf(mx, s[r]);
        }
        mx = max_halves(mx);
        const float m_tile = mx * a.c;   // every tile holds a valid position
        if (__builtin_amdgcn_ballot_w64(m_tile > m_trig)) {
            // acc already holds tile j-1, weighted with the old maximum
            const float m_new = fmaxf(m_run, m_tile);
            const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
            // block by block through vector registers: the accumulator
            // stays in the matrix-core registers everywhere else
#pragma unroll
            for (int db = 0; db < DBV; ++db) {
                f32x16 t = acc_o[db];
                asm volatile("" : "+v"(t));
                t *= alpha;
                asm volatile("" : "+v"(t));
                acc_o[db] = t;
                asm volatile("" : "+a"(acc_o[db]));
            }
        }
        float rowsum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
            float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], a.c, -m_run));
            float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r + 1], a.c, -m_run));
            if (MASKED) {
                p0 = s[r] == -INFINITY ? 0.f : p0;
                p1 = s[r + 1] == -INFINITY ? 0.f : p1;
            }
            rowsum += p0 + p1;
            pk[r >> 1] = pack_bf16(p0, p1);
        }
        l_run += rowsum;
        // the level for the next tile (l = 0 gives m itself)
        m_trig = m_run + fminf(RESCALE_SLACK,
                               fmaxf(0.f, RAISE_SHARE_LOG2 + __builtin_amdgcn_logf(l_run)));

        // tile j+1 must have landed (tiles j+2 and j+3 may stay in flight)
        wait_dma_tiles_left(min(2, max(0, j_hi - 1 - (j + 1))));
        __syncthreads();
    }
};

// Workgroup id -> (batch, latent head, head block, split), laid out so that
// each XCD gets a contiguous range of logical ids (the head blocks and
// splits of one batch element's cache run on one XCD).
__device__ __forceinline__ void decode_wg(const MArgs &a, int bid, int &b, int &hk, int &hblk,
                                          int &split)
{
    const int per = a.n_wg / NXCD, rem = a.n_wg % NXCD;
    const int xcd = bid % NXCD, idx = bid / NXCD;
    int l = xcd * per + (xcd < rem ? xcd : rem) + idx;
    hblk = l % a.n_hblk;
    l /= a.n_hblk;
    split = l % a.n_split;
    l /= a.n_split;
    hk = l % a.Hkv;
    b = l / a.Hkv;
}

// The tile loop of one wave, KH = its k-half (wave-uniform).  Four
// buffers in a ring: tile j lives in buffer (j - j_lo) % 4; tile j+3 goes
// into the buffer of tile j-1 once every wave has done that tile's P V.  The
// ring is unrolled by four so that every buffer reference is static; the
// last tile's P V follows the loop.
template <int KH>
__device__ __forceinline__ void run_tiles(Mla &k, int j_lo, int j_hi, int j_full,
                                          unsigned char *const (&lat)[4],
                                          unsigned char *const (&rot)[4], Xchg &xchg)
{
    uint32_t pk[8];
    int j = j_lo;
    // first tile: nothing before it to multiply into the output
    if (j < j_full)
        k.template step<false, KH, false>(j, j_hi, lat[0], rot[0], lat[3], rot[3], pk, xchg);
    else
        k.template step<true, KH, false>(j, j_hi, lat[0], rot[0], lat[3], rot[3], pk, xchg);
    ++j;
    int u = 1;   // buffer of tile j
    if (j + 2 < j_full) {
        for (; j + 3 < j_full; j += 4) {
            k.template step<false, KH, true>(j, j_hi, lat[1], rot[1], lat[0], rot[0], pk, xchg);
            k.template step<false, KH, true>(j + 1, j_hi, lat[2], rot[2], lat[1], rot[1], pk, xchg);
            k.template step<false, KH, true>(j + 2, j_hi, lat[3], rot[3], lat[2], rot[2], pk, xchg);
            k.template step<false, KH, true>(j + 3, j_hi, lat[0], rot[0], lat[3], rot[3], pk, xchg);
        }
    }
    // at most three full tiles and a ragged one remain; tile j is in buffer
    // (j - j_lo) % 4
    u = (j - j_lo) & 3;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        if (j >= j_hi)
            break;
        // (buffers indexed at run time here: these remaining tiles are few)
        switch (u) {
#define TA_MLA_STEP(U)                                                                          \
    case U:                                                                                     \
        if (j < j_full)                                                                         \
            k.template step<false, KH, true>(j, j_hi, lat[U], rot[U], lat[(U + 3) % 4],          \
                                             rot[(U + 3) % 4], pk, xchg);                        \
        else                                                                                    \
            k.template step<true, KH, true>(j, j_hi, lat[U], rot[U], lat[(U + 3) % 4],           \
                                            rot[(U + 3) % 4], pk, xchg);                         \
        break;
            TA_MLA_STEP(0)
            TA_MLA_STEP(1)
            TA_MLA_STEP(2)
            TA_MLA_STEP(3)
#undef TA_MLA_STEP
        }
        ++j;
        u = (u + 1) & 3;
    }
    // the last tile's P V (its buffer is that of tile j_hi - 1)
    switch ((j_hi - 1 - j_lo) & 3) {
    case 0: k.pv(pk, lat[0]); break;
    case 1: k.pv(pk, lat[1]); break;
    case 2: k.pv(pk, lat[2]); break;
    default: k.pv(pk, lat[3]); break;
    }
}

__global__ __launch_bounds__(NT, 1) void mla_decode_kernel(MArgs args)
{
    __shared__ __attribute__((aligned(16))) unsigned char lat0[LAT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char lat1[LAT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char lat2[LAT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char lat3[LAT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char rot0[ROT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char rot1[ROT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char rot2[ROT_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char rot3[ROT_BYTES];
    __shared__ Xchg xchg;

    Mla k(args);
    const MArgs &a = args;
    const int tid = threadIdx.x;
    k.wave = tid >> 6;
    k.lane = tid & 63;
    k.col = k.lane & 31;
    k.half = k.lane >> 5;
    k.k_half = k.wave & 1;
    k.dim_half = k.wave & 1;

    int b, hk, hblk, split;
    decode_wg(a, blockIdx.x, b, hk, hblk, split);
    const int n_tiles = (a.Skv + BN - 1) / BN;
    const int j_lo = split * a.split_tiles;
    const int j_hi = min(n_tiles, j_lo + a.split_tiles);   // non-empty: splits cover the tiles

    // this lane's head: local index within the latent head's group (the
    // pair of waves 2p, 2p+1 shares heads 32p .. 32p+31 of the block)
    const int h_loc = hblk * HB + (k.wave >> 1) * 32 + k.col;
    const bool head_ok = h_loc < a.g;
    const int head = hk * a.g + min(h_loc, a.g - 1);

    k.kv_b = a.KV + ((size_t)b * a.Skv * a.Hkv + hk) * DL;
    k.kpe_b = a.Kpe + ((size_t)b * a.Skv * a.Hkv + hk) * DR;
    k.init_dma();

    // this wave's half of the query of the lane's head as the B operand:
    // k-step kk holds dims 16kk + 8half .. +8 of [q | q_pe]
    {
        const uint16_t *qp = a.Q + ((size_t)b * a.H + head) * DL + 8 * k.half;
        const uint16_t *qr = a.Qpe + ((size_t)b * a.H + head) * DR + 8 * k.half;
#pragma unroll
        for (int i = 0; i < KKH; ++i) {
            const int kk = k.k_half * KKH + i;
            u32x4 v = kk < KKL ? *(const u32x4 *)(qp + 16 * kk)
                               : *(const u32x4 *)(qr + 16 * (kk - KKL));
            if (!head_ok)
                v = u32x4{0u, 0u, 0u, 0u};
            k.qreg[i] = __builtin_bit_cast(bf16x8, v);
        }
    }
#pragma unroll
    for (int db = 0; db < DBV; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            k.acc_o[db][r] = 0.f;
    k.m_run = -INFINITY;
    k.l_run = 0.f;
    k.m_trig = -INFINITY;

    // prologue: tiles j_lo .. j_lo+2 in flight, wait for the first
    k.dma_tile(j_lo, lat0, rot0);
    if (j_lo + 1 < j_hi)
        k.dma_tile(j_lo + 1, lat1, rot1);
    if (j_lo + 2 < j_hi)
        k.dma_tile(j_lo + 2, lat2, rot2);
    wait_dma_tiles_left(min(2, j_hi - 1 - j_lo));
    __syncthreads();

    // every tile but a ragged last one is fully valid
    const int j_full = min(j_hi, a.Skv / BN);
    unsigned char *const lat[4] = {lat0, lat1, lat2, lat3};
    unsigned char *const rot[4] = {rot0, rot1, rot2, rot3};
    if (k.k_half)
        run_tiles<1>(k, j_lo, j_hi, j_full, lat, rot, xchg);
    else
        run_tiles<0>(k, j_lo, j_hi, j_full, lat, rot, xchg);

    // epilogue: normalise and store this wave's 256 dims of the split's
    // result for the lane's head (both waves of the pair hold the same sums)
    const float l = sum_halves(k.l_run);
    if (head_ok) {
        const float inv = 1.f / l;
        const size_t row = (size_t)b * a.H + head;
        float *op = a.O + (size_t)split * a.o_split + row * DL + DH * k.dim_half;
#pragma unroll
        for (int db = 0; db < DBV; ++db)
#pragma unroll
            for (int gr = 0; gr < 4; ++gr) {
                float4 v;
                v.x = k.acc_o[db][4 * gr + 0] * inv;
                v.y = k.acc_o[db][4 * gr + 1] * inv;
                v.z = k.acc_o[db][4 * gr + 2] * inv;
                v.w = k.acc_o[db][4 * gr + 3] * inv;
                *(float4 *)(op + 32 * db + 8 * gr + 4 * k.half) = v;
            }
        if (k.half == 0 && k.dim_half == 0)
            a.LSE[(size_t)split * a.l_split + row] = (k.m_run + log2f(l)) * LN2;
    }
}

bool overlaps(const void *p, size_t pn, const void *q, size_t qn)
{
    const uintptr_t x = (uintptr_t)p, y = (uintptr_t)q;
    return x < y + qn && y < x + pn;
}

bool misaligned(const void *p) { return ((uintptr_t)p & 15u) != 0; }

constexpr int MAX_SPLITS = 128;
// split heuristic: one workgroup per CU (256 CUs; a workgroup fills its CU's
// register file), at least 8 cache tiles (256 positions) per split
constexpr int64_t MLA_TARGET_WG = 256;
constexpr int MLA_MIN_TILES = 8;

void mla_split_shape(int Skv, int num_splits, int *split_tiles, int *n_split)
{
    const int n_tiles = (Skv + BN - 1) / BN;
    const int per = (n_tiles + num_splits - 1) / num_splits;
    *split_tiles = per;
    *n_split = (n_tiles + per - 1) / per;
}

size_t mla_ws_bytes(int B, int H, int num_splits)
{
    return (size_t)num_splits * B * H * (size_t)(DL + 1) * 4;
}

}  // namespace

extern "C" {

ta_status mla_decode(const void *Q, const void *Q_pe, const void *KV, const void *K_pe,
                     float *O, float *LSE, int B, int H, int Hkv, int Skv, int Dl, int Dr,
                     float scale, int num_splits, void *workspace, size_t workspace_bytes,
                     void *stream)
{
    if (!Q || !Q_pe || !KV || !K_pe || !O || !LSE)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || H < 1 || Hkv < 1 || Skv < 1 || H % Hkv != 0)
        return TA_ERR_INVALID_SHAPE;
    if (num_splits < 1 || num_splits > MAX_SPLITS)
        return TA_ERR_INVALID_SHAPE;
    if (Dl != DL || Dr != DR)
        return TA_ERR_UNSUPPORTED;
    int split_tiles, n_split;
    mla_split_shape(Skv, num_splits, &split_tiles, &n_split);
    const int g = H / Hkv;
    const int n_hblk = (g + HB - 1) / HB;
    const int64_t n_wg = (int64_t)B * Hkv * n_hblk * n_split;
    // 32-bit in-kernel offsets within one tile; 32-bit grid
    if (n_wg >= (1ll << 31) || (int64_t)BN * Hkv * DL * 2 >= (1ll << 31))
        return TA_ERR_INVALID_SHAPE;
    if (misaligned(Q) || misaligned(Q_pe) || misaligned(KV) || misaligned(K_pe) ||
        misaligned(O) || misaligned(LSE))
        return TA_ERR_MISALIGNED;
    if (!(scale >= 0.f) || !isfinite(scale))
        return TA_ERR_INVALID_SCALE;
    const size_t rows = (size_t)B * H;
    const size_t nq = rows * DL, nqr = rows * DR;
    const size_t nkv = (size_t)B * Skv * Hkv * DL, nkr = (size_t)B * Skv * Hkv * DR;
    const size_t o_bytes = nq * 4, l_bytes = rows * 4;
    const void *ins[4] = {Q, Q_pe, KV, K_pe};
    const size_t in_bytes[4] = {nq * 2, nqr * 2, nkv * 2, nkr * 2};
    for (int i = 0; i < 4; ++i)
        if (overlaps(O, o_bytes, ins[i], in_bytes[i]) || overlaps(LSE, l_bytes, ins[i], in_bytes[i]))
            return TA_ERR_ALIASING;
    if (overlaps(O, o_bytes, LSE, l_bytes))
        return TA_ERR_ALIASING;
    const size_t need = n_split > 1 ? mla_ws_bytes(B, H, n_split) : 0;
    if (n_split > 1) {
        if (!workspace || workspace_bytes < need)
            return TA_ERR_WORKSPACE;
        if (misaligned(workspace))
            return TA_ERR_MISALIGNED;
        for (int i = 0; i < 4; ++i)
            if (overlaps(workspace, need, ins[i], in_bytes[i]))
                return TA_ERR_ALIASING;
        if (overlaps(workspace, need, O, o_bytes) || overlaps(workspace, need, LSE, l_bytes))
            return TA_ERR_ALIASING;
    }

    MArgs a;
    a.Q = (const uint16_t *)Q;
    a.Qpe = (const uint16_t *)Q_pe;
    a.KV = (const uint16_t *)KV;
    a.Kpe = (const uint16_t *)K_pe;
    a.B = B;
    a.H = H;
    a.Hkv = Hkv;
    a.Skv = Skv;
    a.g = g;
    a.n_hblk = n_hblk;
    a.n_split = n_split;
    a.split_tiles = split_tiles;
    a.n_wg = (int)n_wg;
    a.c = scale * LOG2E;
    // split partial results: O then LSE of every split (no workspace for one split)
    float *Op = (float *)workspace;
    float *Lp = n_split > 1 ? Op + (size_t)n_split * nq : nullptr;
    if (n_split > 1) {
        a.O = Op;
        a.LSE = Lp;
        a.o_split = nq;
        a.l_split = rows;
    } else {
        a.O = O;
        a.LSE = LSE;
        a.o_split = 0;
        a.l_split = 0;
    }
    hipStream_t s = (hipStream_t)stream;
    hipLaunchKernelGGL(mla_decode_kernel, dim3(a.n_wg), dim3(NT), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && n_split > 1)
        e = tileattn_detail::launch_combine<DL, false>(Op, Lp, O, LSE, (int)rows, n_split, nq,
                                                       rows, s);
    return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH;
}

ta_status mla_workspace_bytes(int B, int H, int num_splits, size_t *bytes)
{
    if (!bytes)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || H < 1 || num_splits < 1 || num_splits > MAX_SPLITS)
        return TA_ERR_INVALID_SHAPE;
    *bytes = num_splits > 1 ? mla_ws_bytes(B, H, num_splits) : 0;
    return TA_OK;
}

ta_status mla_split_heuristic(int B, int H, int Hkv, int Skv, int *num_splits)
{
    if (!num_splits)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || H < 1 || Hkv < 1 || Skv < 1 || H % Hkv != 0)
        return TA_ERR_INVALID_SHAPE;
    const int64_t wg = (int64_t)B * Hkv * (((int64_t)(H / Hkv) + HB - 1) / HB);
    const int n_tiles = (Skv + BN - 1) / BN;
    int n = 1;
    if (wg < MLA_TARGET_WG) {
        n = (int)((MLA_TARGET_WG + wg - 1) / wg);
        n = n < n_tiles / MLA_MIN_TILES ? n : n_tiles / MLA_MIN_TILES;
        n = n < MAX_SPLITS ? n : MAX_SPLITS;
        n = n > 1 ? n : 1;
    }
    *num_splits = n;
    return TA_OK;
}

}  // extern "C"
