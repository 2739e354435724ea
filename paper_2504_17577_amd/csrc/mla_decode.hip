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
//  * One workgroup of eight wave64s (two per SIMD) owns HB = 128 query
//    heads of one latent head of one batch element, and one range of cache
//    tiles (a key split); wave w owns 16 of the heads.  S^T = K Q^T with
//    v_mfma_f32_16x16x32_bf16 over the full 576-wide contraction (A = 16
//    cache rows from LDS, B = the query of the wave's 16 heads, held in
//    registers for the whole kernel: 72 per lane).  In the 16x16 accumulator
//    layout lane l owns head l % 16 and four positions of each 16-position
//    block, so the softmax row reductions are in-lane plus two lane swaps
//    (v_permlane32_swap, v_permlane16_swap).  No wave shares its scores or
//    its softmax with another.
//  * O^T += V^T P^T over all 512 output dims of the wave's heads (32 blocks
//    of 16 dims, 128 fp32 registers per lane): the bf16 weights already sit
//    in the B-operand layout (the MFMA's 32-position reduction order is
//    chosen to match), and V^T comes from the same latent rows in LDS through
//    the transpose read ds_read_b64_tr_b16.  The P V of tile j-1 is issued
//    among the score MFMAs of tile j (alternately), and the 68 MFMAs of a
//    tile run as one software pipeline whose LDS operands are read three
//    MFMAs ahead (with
//    every register given to the query and the accumulator, the compiler's
//    own schedule read each operand just before its MFMA and waited for it).
//  * Cache tiles of 32 positions go global -> LDS by DMA (buffer_load_dwordx4
//    ... lds) into a ring of four buffers, two tiles ahead of the one in
//    use: the latent part [32][512] and the rotary part [32][64] of a tile
//    side by side; one barrier per tile.  16-byte chunks are XOR-swizzled so
//    that the score operand reads (ds_read_b128) and the transpose reads of
//    the same latent rows are both bank-conflict free (chunk c of latent row
//    r at c ^ (2 (r & 7) + ((r >> 3) & 1)) within its aligned group of 16,
//    of rotary row r at c ^ ((r >> 1) & 7)): a score operand read touches
//    rows 16b .. 16b + 15 at one chunk each, a transpose read rows 4g .. 4g + 3
//    of two lane groups at two adjacent chunks each.
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
#include "lds_dma.h"
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
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;

constexpr int DL = 512;              // latent width (query, cache, output)
constexpr int DR = 64;               // rotary width (query, key)
constexpr int BN = 32;               // cache positions per tile
constexpr int NW = 8;                // waves per workgroup (two per SIMD)
constexpr int NT = 64 * NW;          // threads per workgroup
constexpr int HW = 16;               // query heads per wave
constexpr int HB = HW * NW;          // query heads per workgroup
constexpr int KSL = DL / 32;         // MFMA k-steps (32 wide) over the latent part
constexpr int KS = (DL + DR) / 32;   // ... over latent and rotary
constexpr int DBO = DL / 16;         // 16-row blocks of a wave's O^T
constexpr int LAT_BYTES = BN * DL * 2;
constexpr int ROT_BYTES = BN * DR * 2;
constexpr int STAGE_BYTES = LAT_BYTES + ROT_BYTES;
constexpr int NST = 4;               // ring buffers
constexpr int PF = 3;                // MFMA operands read ahead of their MFMA
constexpr int LAT_PER_THREAD = BN * (DL / 8) / NT;   // 16-byte latent DMA chunks per thread
constexpr int ROT_THREADS = BN * (DR / 8);           // threads with one rotary chunk each
constexpr int NXCD = 8;
constexpr float LOG2E = 1.44269504088896340736f;
constexpr float LN2 = 0.69314718055994530942f;
constexpr float RESCALE_SLACK = 8.0f;       // base-2 headroom: weights never exceed 2^8
constexpr float RAISE_SHARE_LOG2 = -2.0f;   // log2 of the share (1/4) of l a position may
                                            // weigh before the max is raised
static_assert(KSL == 16 && KS == 18 && DBO == 32, "k-steps / output blocks");
static_assert(LAT_PER_THREAD == 4 && ROT_THREADS == 256 && NT == 512, "tile/thread mismatch");

typedef float f32x4 __attribute__((ext_vector_type(4)));

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
__device__ __forceinline__ int lat_swz(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }
__device__ __forceinline__ int rot_swz(int r) { return (r >> 1) & 7; }

__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// x over the four lanes l, l ^ 16, l ^ 32, l ^ 48 that hold one head
__device__ __forceinline__ float max_head(float x)
{
    u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                               false);
    x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float sum_head(float x)
{
    u32x2 r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                               false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Tile DMA is issued as inline assembly (lds_dma.h), so the compiler does
// not track it: it never drains the tile loads in flight at a barrier, and
// the kernel waits for them itself.  The kernel's only other vector-memory
// operations are the query loads, waited for before the first tile, and the
// output stores after the last tile.  Waves 0-3 issue one rotary chunk per
// tile besides their latent chunks.
template <int TILES_IN_FLIGHT>
__device__ __forceinline__ void wait_tiles(bool rot_wave)
{
    if (rot_wave)
        tileattn_dma::wait_vmcnt<TILES_IN_FLIGHT * (LAT_PER_THREAD + 1)>();
    else
        tileattn_dma::wait_vmcnt<TILES_IN_FLIGHT * LAT_PER_THREAD>();
}

struct Mla {
    const MArgs &a;
    int wave, lane, hc, gq;         // hc = lane % 16 (the head), gq = lane / 16
    int wave_u;                     // the wave index, in a scalar register
    bool rot_wave;                  // this wave also fetches rotary chunks
    bool busy;                      // some of this wave's 16 heads exist (else it only
                                    // takes part in the tile DMA and the barriers)
    const uint16_t *kv_b, *kpe_b;   // cache of (batch, latent head) at position 0
    uint32_t lat_off[2], rot_off;   // per-lane DMA source offsets (see init_lanes)
    uint32_t ka0, ra0;              // per-lane LDS offsets of the score operands
    uint32_t va0;                   // ... of the value transpose reads
    bf16x8 qreg[KS];                // the query of head hc: dims 32kk + 8gq .. +8
    f32x4 acc_o[DBO];
    float m_run, l_run;
    float m_trig;   // the running max is raised when a tile max exceeds this

    __device__ Mla(const MArgs &args) : a(args) {}

    // Latent DMA slot i*NT + 64w + l (i < 4) is row r = 8i + w, stored chunk
    // l, fetched from source chunk l ^ lat_swz(r) = l ^ (2w + (i & 1)): two
    // per-lane offsets (rows w and 8 + w) and a scalar 16 (i >> 1) rows of
    // pitch address all four.  Rotary slot 64w + l (waves 0-3) is row
    // 8w + l / 8, chunk l % 8, fetched from chunk (l % 8) ^ rot_swz(row).
    //   Score operand of k-step kk, position block b (rows 16b + hc): latent
    // chunk 4kk + gq at byte 256 (kk >> 2) + 16 ((4 (kk & 3) + gq) ^ lat_swz(hc))
    // of the row, rotary chunk 4 (kk - 16) + gq at 16 ((4 (kk - 16) + gq) ^
    // (hc >> 1)).
    //   Value transpose reads: in each group of 16 lanes, lane 4i + c reads
    // dims d0 + 4c .. +3 of row r0 + i, and lane j of the group then holds dim
    // d0 + j of rows r0 .. r0 + 3.  Group gq reads rows 4gq .. (k-slots 0-3)
    // and 16 + 4gq .. (k-slots 4-7, the same swizzle 16 KiB on); dims
    // 16db .. of block db are chunk 2db + ((hc & 3) >> 1), byte 8 (hc & 1).
    __device__ __forceinline__ void init_lanes()
    {
        const uint32_t lat_pitch = (uint32_t)a.Hkv * DL * 2, rot_pitch = (uint32_t)a.Hkv * DR * 2;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int r = 8 * p + wave_u;
            lat_off[p] = r * lat_pitch + 16 * (lane ^ lat_swz(r));
        }
        const int rr = 8 * (wave_u & 3) + lane / 8;
        rot_off = rr * rot_pitch + 16 * ((lane % 8) ^ rot_swz(rr));
        ka0 = hc * (DL * 2) + 16 * (gq ^ lat_swz(hc));
        ra0 = LAT_BYTES + hc * (DR * 2) + 16 * (gq ^ (hc >> 1));
        const int row = 4 * gq + (hc >> 2);
        va0 = row * (DL * 2) + 16 * (((hc & 3) >> 1) ^ lat_swz(row)) + 8 * (hc & 1);
    }

    // DMA cache tile j (positions j*BN ..) into `stage`, with non-temporal
    // loads: each tile is read by this workgroup only, once (measured 1-2.5 %
    // faster on mla_b64_s8k and mla_b128_s4k, the same output).  Each buffer
    // resource starts at the tile and ends after its last valid row; a row
    // past Skv re-reads the last valid row (its scores are masked and its
    // weights zero), so no lane addresses outside the cache.
    __device__ __forceinline__ void dma_tile(int j, unsigned char *stage) const
    {
        const int valid = min(BN, a.Skv - j * BN);
        const size_t row0 = (size_t)j * BN * a.Hkv;
        const uint32_t lat_pitch = (uint32_t)a.Hkv * DL * 2, rot_pitch = (uint32_t)a.Hkv * DR * 2;
        const tileattn_dma::u32x4s rl =
            tileattn_dma::buffer_rsrc(kv_b + row0 * DL, (valid - 1) * lat_pitch + DL * 2);
        const uint32_t lat_base = tileattn_dma::lds_addr(stage) + wave_u * 64 * 16;
        if (valid == BN) {
#pragma unroll
            for (int i = 0; i < LAT_PER_THREAD; ++i)
                tileattn_dma::dma16_soff<true>(lat_base + i * NT * 16, lat_off[i & 1],
                                         16 * (i >> 1) * lat_pitch, rl);
        } else {
            const int last = valid - 1;
#pragma unroll
            for (int i = 0; i < LAT_PER_THREAD; ++i) {
                // row 8i + w, or the last valid row past it (the difference,
                // possibly negative, is added modulo 2^32)
                const int row = 8 * i + wave_u;
                const int src = row > last ? last : row;
                const uint32_t o = lat_off[i & 1] + (uint32_t)((src - 8 * (i & 1) - wave_u) *
                                                               (int)lat_pitch);
                tileattn_dma::dma16<true>(lat_base + i * NT * 16, o, rl);
            }
        }
        if (rot_wave) {
            const tileattn_dma::u32x4s rr =
                tileattn_dma::buffer_rsrc(kpe_b + row0 * DR, (valid - 1) * rot_pitch + DR * 2);
            // row 8w + l/8 is lane-dependent: clamp per lane
            const int row = 8 * (wave_u & 3) + lane / 8;
            const int shift = row > valid - 1 ? row - (valid - 1) : 0;
            tileattn_dma::dma16<true>(tileattn_dma::lds_addr(stage + LAT_BYTES) + wave_u * 64 * 16,
                                rot_off - (uint32_t)shift * rot_pitch, rr);
        }
    }

    // The tile's MFMA work as one software pipeline: the score MFMAs of the
    // tile in `ss` (S^T[position][head] of its two 16-position blocks, 18
    // k-steps each, SC) and the P V of the previous tile, whose rows are in
    // `sv` and whose weights are pk (PV), issued alternately while both
    // remain (a score MFMA's operand is one ds_read_b128, a P V MFMA's two
    // transpose reads: mixed, the two kinds of read keep the LDS busier than
    // in two separate phases).  Each MFMA's LDS operand is read PF MFMAs
    // ahead, and scheduling barriers keep that order, so the LDS latency is
    // covered by the MFMAs in between.
    //   P V: O^T += V^T P^T over all 512 dims; the weights pk are in the
    // B-operand layout (k-slot t of lane group gq is position 4gq + t for
    // t < 4, 16 + 4gq + t - 4 after), V^T comes through the transpose reads.
    template <bool SC, bool PV>
    __device__ __forceinline__ void mma(const unsigned char *ss, const unsigned char *sv,
                                        f32x4 (&s)[2], const uint32_t (&pk)[4])
    {
        constexpr int NS = SC ? 2 * KS : 0;
        constexpr int N = NS + (PV ? DBO : 0);
        const bf16x8 bv = __builtin_bit_cast(bf16x8, u32x4{pk[0], pk[1], pk[2], pk[3]});
        // The operand offsets of chunk index c ^ swizzle differ from those of
        // c = 0 in the XOR of c's own bits (the swizzle and the row base
        // occupy other bits), and the ring is aligned so that adding a stage
        // base keeps that true: the latent score operand of k-step 4q + m is
        // at (ka0 ^ 64m) + 256q, the rotary one of k-step 16 + m at ra0 ^ 64m,
        // the value rows of block 8g + m at (va0 ^ 32m) + 256g.
        const uint32_t kb = tileattn_dma::lds_addr(ss) + ka0;
        const uint32_t rb = tileattn_dma::lds_addr(ss) + ra0;
        const uint32_t vb = tileattn_dma::lds_addr(sv) + va0;
        // Items i < NS are score MFMAs: k-step kk_of(i) of position block
        // i & 1; items NS + v are P V MFMAs of output block db_of(v).  Both
        // orders keep m, the XOR term, fixed for four items in a row.
        auto kk_of = [](int i) {
            const int u = i >> 1;   // 0 .. 17
            return u < KSL ? 4 * (u & 3) + (u >> 2) : u;
        };
        auto db_of = [](int v) { return 8 * (v & 3) + (v >> 2); };
        auto operand = [&](int i) -> bf16x8 {
            if (i < NS) {
                const int kk = kk_of(i), b = i & 1;
                const uint32_t p = kk < KSL
                    ? (kb ^ (64u * (kk & 3))) + 256u * (kk >> 2) + 16u * (DL * 2) * b
                    : (rb ^ (64u * (kk - KSL))) + 16u * (DR * 2) * b;
                return *(const lds_bf16x8 *)(uintptr_t)p;
            }
            const int db = db_of(i - NS);
            const uint32_t p = (vb ^ (32u * (db & 7))) + 256u * (db >> 3);
            const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(uintptr_t)p);
            const i16x4 hi =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(uintptr_t)(p + 16u * (DL * 2)));
            const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
            return __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
        };
        if (SC) {
            s[0] = f32x4{0.f, 0.f, 0.f, 0.f};
            s[1] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        // issue order: score and P V items alternate while both remain
        constexpr int NPV = N - NS;
        auto item = [](int x) {
            if (NS == 0 || NPV == 0)
                return x;
            const int m2 = NPV < NS ? NPV : NS;
            if (x < 2 * m2)
                return (x & 1) ? NS + (x >> 1) : (x >> 1);
            return NS > NPV ? x - m2 : NS + (x - m2);
        };
        bf16x8 buf[PF];
#pragma unroll
        for (int i = 0; i < PF; ++i)
            if (i < N)
                buf[i] = operand(item(i));
#pragma unroll
        for (int x = 0; x < N; ++x) {
            __builtin_amdgcn_sched_barrier(0);
            const int i = item(x);
            if (i < NS)
                s[i & 1] = mfma16(buf[x % PF], qreg[kk_of(i)], s[i & 1]);
            else
                acc_o[db_of(i - NS)] = mfma16(buf[x % PF], bv, acc_o[db_of(i - NS)]);
            if (x + PF < N)
                buf[x % PF] = operand(item(x + PF));
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    // Online softmax of tile j: mask, running max, weights into pk
    template <bool MASKED>
    __device__ __forceinline__ void softmax(int j, f32x4 (&s)[2], uint32_t (&pk)[4])
    {
        // lane holds positions j*BN + 16b + 4gq + r of head hc
        float mx = -INFINITY;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (MASKED) {
                    const int pos = j * BN + 16 * b + 4 * gq + r;
                    s[b][r] = pos < a.Skv ? s[b][r] : -INFINITY;
                }
                mx = fmaxf(mx, s[b][r]);
            }
        mx = max_head(mx);
        const float m_tile = mx * a.c;   // every tile holds a valid position
        if (__builtin_amdgcn_ballot_w64(m_tile > m_trig)) {
            // acc holds the tiles before j (once their MFMAs are done),
            // weighted with the old maximum
            const float m_new = fmaxf(m_run, m_tile);
            const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DBO; ++db)
                acc_o[db] *= alpha;
        }
        float rowsum = 0.f;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 4; r += 2) {
                float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][r], a.c, -m_run));
                float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][r + 1], a.c, -m_run));
                if (MASKED) {
                    p0 = s[b][r] == -INFINITY ? 0.f : p0;
                    p1 = s[b][r + 1] == -INFINITY ? 0.f : p1;
                }
                rowsum += p0 + p1;
                pk[2 * b + (r >> 1)] = pack_bf16(p0, p1);
            }
        l_run += rowsum;
        // the level for the next tile (l = 0 gives m itself)
        m_trig = m_run + fminf(RESCALE_SLACK,
                               fmaxf(0.f, RAISE_SHARE_LOG2 + __builtin_amdgcn_logf(l_run)));
    }

    // Tile t (counted from the split's first, key tile j = j_lo + t) in
    // stage t % 4: once it has landed and every wave is past tile t-1, tile
    // t+2 goes into the stage of tile t-2; then the scores of tile t, the
    // P V of tile t-1 (weights pk, rows in stage (t-1) % 4) and the softmax
    // of tile t, whose weights replace pk.
    template <bool MASKED, bool FIRST>
    __device__ __forceinline__ void step(int t, int n, int j_lo, unsigned char *ring,
                                         uint32_t (&pk)[4])
    {
        if (t + 1 < n)
            wait_tiles<1>(rot_wave);
        else
            wait_tiles<0>(rot_wave);
        __syncthreads();
        if (t + 2 < n)
            dma_tile(j_lo + t + 2, ring + ((t + 2) % NST) * STAGE_BYTES);
        if (busy) {
            f32x4 s[2];
            mma<true, !FIRST>(ring + (t % NST) * STAGE_BYTES,
                              ring + ((t + NST - 1) % NST) * STAGE_BYTES, s, pk);
            softmax<MASKED>(j_lo + t, s, pk);
        }
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

__global__ __launch_bounds__(NT, 1) void mla_decode_kernel(MArgs args)
{
    __shared__ __attribute__((aligned(1024))) unsigned char ring[NST * STAGE_BYTES];

    Mla k(args);
    const MArgs &a = args;
    const int tid = threadIdx.x;
    k.wave = tid >> 6;
    k.lane = tid & 63;
    k.hc = k.lane & 15;
    k.gq = k.lane >> 4;
    k.wave_u = __builtin_amdgcn_readfirstlane(k.wave);
    k.rot_wave = k.wave_u < ROT_THREADS / 64;

    int b, hk, hblk, split;
    decode_wg(a, blockIdx.x, b, hk, hblk, split);
    const int n_tiles = (a.Skv + BN - 1) / BN;
    const int j_lo = split * a.split_tiles;
    const int j_hi = min(n_tiles, j_lo + a.split_tiles);   // non-empty: splits cover the tiles
    const int n = j_hi - j_lo;

    // this lane's head: local index within the latent head's group
    const int h_loc = hblk * HB + k.wave_u * HW + k.hc;
    const bool head_ok = h_loc < a.g;
    const int head = hk * a.g + min(h_loc, a.g - 1);
    k.busy = hblk * HB + k.wave_u * HW < a.g;   // wave-uniform

    k.kv_b = a.KV + ((size_t)b * a.Skv * a.Hkv + hk) * DL;
    k.kpe_b = a.Kpe + ((size_t)b * a.Skv * a.Hkv + hk) * DR;
    k.init_lanes();

    // prologue: the first two tiles in flight
    k.dma_tile(j_lo, ring);
    if (n > 1)
        k.dma_tile(j_lo + 1, ring + STAGE_BYTES);

    // the query of the lane's head as the B operand: k-step kk holds dims
    // 32kk + 8gq .. +8 of [q | q_pe]
    {
        const uint16_t *qp = a.Q + ((size_t)b * a.H + head) * DL + 8 * k.gq;
        const uint16_t *qr = a.Qpe + ((size_t)b * a.H + head) * DR + 8 * k.gq;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            u32x4 v = kk < KSL ? *(const u32x4 *)(qp + 32 * kk)
                               : *(const u32x4 *)(qr + 32 * (kk - KSL));
            if (!head_ok)
                v = u32x4{0u, 0u, 0u, 0u};
            k.qreg[kk] = __builtin_bit_cast(bf16x8, v);
        }
    }
#pragma unroll
    for (int db = 0; db < DBO; ++db)
        k.acc_o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
    k.m_run = -INFINITY;
    k.l_run = 0.f;
    k.m_trig = -INFINITY;
    // the query (issued after the prologue tiles; the tiles are waited for
    // by the first step)
    tileattn_dma::wait_vmcnt<0>();

    // every tile but a ragged last one is fully valid
    const int n_full = min(j_hi, a.Skv / BN) - j_lo;
    uint32_t pk[4];
    if (n_full > 0)
        k.step<false, true>(0, n, j_lo, ring, pk);
    else
        k.step<true, true>(0, n, j_lo, ring, pk);
    int t = 1;
    for (; t < n_full; ++t)
        k.step<false, false>(t, n, j_lo, ring, pk);
    if (t < n)
        k.step<true, false>(t, n, j_lo, ring, pk);
    // the last tile's P V
    {
        f32x4 s_unused[2];
        if (k.busy)
            k.mma<false, true>(ring, ring + ((n - 1) % NST) * STAGE_BYTES, s_unused, pk);
    }

    // epilogue: normalise and store the split's result of the lane's head:
    // block db, lane group gq holds dims 16db + 4gq .. +3
    const float l = sum_head(k.l_run);
    if (head_ok) {
        const float inv = 1.f / l;
        const size_t row = (size_t)b * a.H + head;
        float *op = a.O + (size_t)split * a.o_split + row * DL + 4 * k.gq;
#pragma unroll
        for (int db = 0; db < DBO; ++db)
            *(f32x4 *)(op + 16 * db) = k.acc_o[db] * inv;
        if (k.gq == 0)
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
