// Fused scaled-dot-product attention forward for gfx950 (MI355X).
//
// One workgroup of four wave64s owns BM = 128 query rows of one (batch, head)
// and streams the key/value sequence through LDS in tiles of BN = 64 keys,
// keeping the softmax state and the output accumulator in registers.  This is
// the tile-fused recurrence of the paper's attention listing (appendix,
// "Implementation of FlashMLA with TileLang"): per key tile, scores, running
// row max, rescale factor exp(m_old - m_new), exponentials, running row sum,
// rescale of the accumulator, accumulate P V; divide by the row sum at the
// end.  The design below is this library's own for CDNA4:
//
//  * Each wave computes S^T = K Q^T for its 32 queries with
//    v_mfma_f32_32x32x16_bf16 (A = K rows from LDS, B = Q held in registers
//    for the whole kernel).  In the 32x32 accumulator layout lane l owns
//    query l % 32, so a row reduction is in-lane plus one v_permlane32_swap.
//  * The same lane ownership carries into O^T = V^T P^T: the exponentials
//    of the scores, rounded to bf16, already sit in the B-operand layout;
//    the order of the 16 keys of each MFMA step is chosen to match, and the
//    A operand (V^T) is read from the row-major V tile with the gfx950 LDS
//    transpose read ds_read_b64_tr_b16, so V needs no reshuffle.  The
//    per-row rescale factor is a per-lane scalar.
//  * K and V tiles go global -> LDS by direct DMA (buffer_load_dwordx4 ...
//    lds, 16 bytes per lane, issued as inline assembly and waited for by
//    the kernel itself), in two stages: the DMA of tile j+1 is issued
//    before the math on tile j, with one barrier per tile.  Each lane
//    fetches the 16-byte chunk that belongs at its LDS slot, which is how
//    the XOR swizzles that keep the MFMA operand reads bank-conflict free
//    are applied.
//  * Two workgroups share each CU (two waves per SIMD), so the MFMAs of one
//    wave overlap the softmax arithmetic of the other.
//  * The running max m is raised (and the accumulator and row sum
//    rescaled) only when a row's tile max passes the level
//    m + min(8, max(0, log2(l / 4))), l being the lane's running row sum.
//    Below that level a new key's weight is at most max(1, l / 4) and 2^8:
//    a key weighted above 1 can end with at most a fifth of its row's mass,
//    so the bf16 rounding of its weight is diluted, while a key that could
//    dominate its row raises the max first and is weighted exactly 1.  In
//    exact arithmetic the result is the same softmax for any level; the
//    level is computed once per tile, off the path from the scores to the
//    rescale decision, and on rows with many comparable keys it rarely
//    triggers after the first tiles.
//  * Causal: key tiles beyond the last visible key of the workgroup are not
//    visited; only tiles crossing the diagonal or the end of the sequence
//    take the masked path; there, waves whose queries see none of a tile
//    skip it.
//  * Epilogue: the normalised O rows are staged in LDS so that each store
//    instruction writes whole rows.
//  * Work items are (batch, head, query tile) triples; the hardware deals
//    consecutive workgroup ids round-robin to the 8 XCDs, so each XCD gets
//    a contiguous range of heads (their K/V stay in that XCD's L2),
//    heaviest causal tiles first.  Non-causal grids (and grids that fit on
//    the chip at once) have one workgroup per item.  Larger causal grids are
//    persistent, two workgroups per CU, each running its items as one
//    stream of key tiles: the next item's first K/V tile and its Q are
//    fetched during the current item's last tile, and the current item's O
//    stores overlap the next item's first tile.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <atomic>

#include "tileattn.h"
#include "lds_dma.h"
#include "split_combine.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(1))) void glb_void;

constexpr int BM = 128;      // query rows per workgroup (4 waves x 32)
constexpr int BM_SMALL = 64; // the same with 16 query rows per wave (small grids)
constexpr int BN = 64;       // keys per tile
constexpr int NT = 256;      // threads per workgroup
constexpr int NXCD = 8;      // XCDs per MI355X
constexpr int PF_S = 4;      // score MFMA operands read ahead of their MFMA
constexpr int PF_V = 3;      // P V MFMA operands read ahead of their MFMA
constexpr float LOG2E = 1.44269504088896340736f;
constexpr float LN2 = 0.69314718055994530942f;
constexpr float RESCALE_SLACK = 8.0f;   // base-2 headroom: weights never exceed 2^8
constexpr float RAISE_SHARE_LOG2 = -2.0f;  // log2 of the share (1/4) of l a key may
                                            // weigh before the max is raised
// word 3 of a raw (unswizzled, stride 0) buffer resource on CDNA: 32-bit
// data format, loads past num_records return zero
[[maybe_unused]] constexpr int BUF_RSRC_WORD3 = 0x00020000;

template <int D>
struct Cfg {
    static constexpr int CH = D / 8;                  // 16-byte chunks per row
    static constexpr int TILE_BYTES = BN * D * 2;     // one K or V tile
    static constexpr int DMA_PER_THREAD = BN * CH / NT;
    static constexpr int DB = D / 32;                 // 32-row blocks of O^T
    static constexpr int KK = D / 16;                 // MFMA k-steps for S^T
    static_assert(BN * CH % NT == 0, "tile/thread mismatch");
    // K tile: 16-byte chunk c of row r lives at chunk c ^ kswz(r); makes the
    // 32-row A-operand reads conflict free
    __device__ static int kswz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
    // V tile: same for the transpose reads (4 rows x 64 bytes per half wave)
    __device__ static int vswz(int r) { return D == 128 ? 4 * (r & 3) : 4 * ((r >> 1) & 1); }
};

struct Args {
    const uint16_t *Q, *K, *V;
    // O: fp32 or bf16 [B, Hq, Sq, D] (per the kernel's OBF16), LSE fp32
    // [B, Hq, Sq].  With key splits these are the partial results of split 0
    // and split s adds s * o_split / s * l_split elements.
    void *O;
    float *LSE;
    size_t o_split, l_split;
    int B, Hq, Hkv, Sq, Sk;
    int group;       // Hq / Hkv
    int n_qt;        // query tiles per head
    int n_split;     // key-range splits per query tile
    int split_tiles; // key tiles per split
    int n_items;     // work items: B * Hq * n_qt * n_split
    int cu_per_xcd;  // CUs of one XCD (0: unknown)
    float c;         // scale * log2(e)
};

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    // one v_cvt_pk_bf16_f32: both halves rounded to nearest even
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// max of x over lanes l and l ^ 32 (the two halves holding one query row)
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

// the same over lanes l and l ^ 16
__device__ __forceinline__ float max_rows16(float x)
{
    const u32x2 r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                     false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float sum_rows16(float x)
{
    const u32x2 r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                     false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Work items are (batch * head, query tile, key split) triples, numbered
// head-major (heaviest causal query tiles of a head first).  The hardware
// hands workgroup w to XCD w % 8, and each XCD owns a contiguous range of
// items, so that a head's K/V stay in that XCD's L2.
__device__ __forceinline__ int xcd_range_lo(const Args &a, int x)
{
    const int per = a.n_items / NXCD, rem = a.n_items % NXCD;
    return x * per + (x < rem ? x : rem);
}

__device__ __forceinline__ int xcd_range_n(const Args &a, int x)
{
    return a.n_items / NXCD + (x < a.n_items % NXCD ? 1 : 0);
}

// Persistent grid: workgroup bid's item of round r (-1 past the end of its
// XCD's range).  The workgroups of an XCD (S of them, slot = bid / 8) take
// its range in rounds of S items, in alternating direction: round r gives
// slot s the item r*S + s (even r) or r*S + S-1-s (odd r).  For causal items
// (heaviest query tiles of a head first) this gives every workgroup about
// the same work over each pair of rounds, and all the workgroups of an XCD
// work on the same one or two heads at a time.
__device__ __forceinline__ int persistent_item(const Args &a, int bid, int grid, int r)
{
    const int xcd = bid % NXCD, slot = bid / NXCD;
    const int S = (grid - xcd + NXCD - 1) / NXCD;
    const int i = r * S + ((r & 1) ? S - 1 - slot : slot);
    return i < xcd_range_n(a, xcd) ? xcd_range_lo(a, xcd) + i : -1;
}

// One workgroup per item: workgroup bid's item.  The hardware fills every CU
// of an XCD with one workgroup (slots 0 .. R-1, R = CUs per XCD) before it
// puts a second one on any (slots R .. 2R-1 again on CUs 0 .. R-1, and so
// on), so the slots are dealt the XCD's items in rounds of R in alternating
// direction: slot k and slot R + k, which share a CU, get a heavy and a
// light causal query tile instead of two alike.
__device__ __forceinline__ int static_item(const Args &a, int bid)
{
    const int xcd = bid % NXCD, slot = bid / NXCD;
    const int n = xcd_range_n(a, xcd);
    const int R = a.cu_per_xcd > 0 ? a.cu_per_xcd : n;
    const int r = slot / R, p = slot % R;
    const int m = min(R, n - r * R);   // slots of this round
    return xcd_range_lo(a, xcd) + r * R + ((r & 1) ? m - 1 - p : p);
}

// One work item's coordinates and key-tile range (wave-uniform).
struct Item {
    int q0;          // first query row
    int split;       // key split index
    int j_lo, j_hi;  // key tiles [j_lo, j_hi) of this item
    int j_fast;      // tiles before this one need no per-element mask
    size_t row0;     // (b * Hq + hq) * Sq: first row of the head in Q, O, LSE
    size_t kv_base;  // (b * Hkv + hk) * Sk * D: the head's K/V slice
};

// QW = 32 or 16 query rows per wave.  QW = 32: S^T and O^T blocks of
// v_mfma_f32_32x32x16_bf16, lane l owns query l % 32 and half l / 32 of
// each block's rows.  QW = 16: blocks of v_mfma_f32_16x16x32_bf16, lane l
// owns query l % 16 and quarter l / 16 (64-query workgroups, for grids
// that leave the CUs short of waves).
template <int D, int QW, bool CAUSAL, bool OBF16, bool PERSIST>
struct Kernel {
    using C = Cfg<D>;
    static constexpr int BMQ = 4 * QW;                     // query rows per workgroup
    static constexpr int NKB = BN / QW;                    // key blocks of a tile
    static constexpr int KK = QW == 32 ? D / 16 : D / 32;  // k-steps of the scores
    static constexpr int DB = D / QW;                      // row blocks of O^T
    static constexpr int NG = 64 / QW;                     // lanes per query
    using Acc = typename std::conditional<QW == 32, f32x16, f32x4>::type;
    static constexpr int AR = QW == 32 ? 16 : 4;           // accumulator values per block

    const Args &a;
    int wave, lane;
    int col, half;           // lane % QW (the query), lane / QW
    int wave_u;              // the wave index, in a scalar register
    int off;                 // Sk - Sq, the bottom-right causal offset
    Item cur, nxt;           // the item being computed and the workgroup's next one
    bool has_next;
    int qi, q_last_wave;     // this lane's query row; last real row of the wave
    bool wave_has_rows;
    uint32_t koff, voff;     // byte offsets of this lane's first K / V chunk in a tile
    bf16x8 qreg[KK];
    Acc acc_o[DB];
    float m_run, l_run;
    float m_trig;   // the running max is raised when a tile max exceeds this

    __device__ Kernel(const Args &args) : a(args) {}

    __device__ __forceinline__ Item describe(int L) const
    {
        const int per_head = PERSIST ? a.n_qt : a.n_qt * a.n_split;
        const int head = L / per_head;
        int qt = PERSIST ? L % per_head : (L % per_head) / a.n_split;
        Item it;
        it.split = PERSIST ? 0 : L % a.n_split;   // persistent grids have no key splits
        if (CAUSAL)
            qt = a.n_qt - 1 - qt;   // heaviest query tiles of a head first
        const int b = head / a.Hq, hq = head % a.Hq;
        const int hk = hq / a.group;
        it.q0 = qt * BMQ;
        it.row0 = ((size_t)b * a.Hq + hq) * a.Sq;
        it.kv_base = ((size_t)b * a.Hkv + hk) * (size_t)a.Sk * D;
        // key tiles to visit, and the first one needing per-element masks
        const int n_kv_all = (a.Sk + BN - 1) / BN;
        int n_kv = n_kv_all;
        int first_masked = (a.Sk % BN) ? n_kv_all - 1 : n_kv_all;
        if (CAUSAL) {
            const int q_last_wg = min(it.q0 + BMQ, a.Sq) - 1;
            n_kv = min(n_kv_all, (q_last_wg + off) / BN + 1);
            first_masked = min(first_masked, max(0, (it.q0 + off + 1) / BN));
            first_masked = min(first_masked, n_kv);
        }
        it.j_lo = PERSIST ? 0 : it.split * a.split_tiles;
        it.j_hi = PERSIST ? n_kv : min(n_kv, it.j_lo + a.split_tiles);
        it.j_fast = min(first_masked, it.j_hi);
        return it;
    }

    // per-lane values of the current item (the per-wave ones from the wave
    // index in a scalar register, so that branches on them are uniform)
    __device__ __forceinline__ void set_rows()
    {
        qi = cur.q0 + wave * QW + col;
        q_last_wave = min(cur.q0 + wave_u * QW + QW - 1, a.Sq - 1);
        wave_has_rows = cur.q0 + wave_u * QW < a.Sq;
    }

    __device__ __forceinline__ void reset_state()
    {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r = 0; r < AR; ++r)
                acc_o[db][r] = 0.f;
        m_run = -INFINITY;
        l_run = 0.f;
        m_trig = -INFINITY;
    }

    // Q of this lane's query of item `it`, as the B operand of S^T = K Q^T.
    // Rows past Sq (padding of the last query tile) read row Sq-1: their
    // results are never stored.
    __device__ __forceinline__ void load_q(const Item &it)
    {
        // (dims 8 NG kk + 8 half .. +7 for k-step kk)
        const int r = min(it.q0 + wave * QW + col, a.Sq - 1);
        const uint16_t *qp = a.Q + (it.row0 + r) * D + 8 * half;
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
            qreg[kk] = __builtin_bit_cast(bf16x8, *(const u32x4 *)(qp + 8 * NG * kk));
    }

    // Each lane's source byte offset (within a tile) for its 16-byte LDS
    // slots: slot i*NT + 64w + l holds chunk (pc ^ swizzle(r)) of tile row r.
    // Row r = i * RPS + (64w + l) / CH, and both swizzles depend on r only
    // through (64w + l) / CH, so slot i's offset is that of slot 0 plus
    // i * NT * 16 bytes (RPS rows).
    __device__ void init_dma()
    {
        wave_u = __builtin_amdgcn_readfirstlane(wave);
        const int slot = wave_u * 64 + lane;
        const int r = slot / C::CH, pc = slot % C::CH;
        koff = 2 * (r * D + 8 * (pc ^ C::kswz(r)));
        voff = 2 * (r * D + 8 * (pc ^ C::vswz(r)));
    }

    // DMA the K or V tile of keys j*BN .. j*BN+BN-1 of the head slice at
    // `base` into LDS at `buf` (buffer_load_dwordx4 ... lds, issued as inline
    // assembly: the compiler does not track these loads, the kernel waits for
    // them itself at the end of every tile).  The buffer resource starts at
    // the tile and ends at the end of the slice; on the ragged last tile rows
    // past Sk re-read row Sk-1 (their scores are masked and their weights
    // zero), so no lane addresses past the slice.
    template <bool IS_V>
    __device__ __forceinline__ void dma_tile(const uint16_t *base, int j,
                                             const unsigned char *buf) const
    {
        constexpr int RPS = NT * 16 / (2 * D);   // tile rows per slot block
        const uint32_t tile_bytes = BN * D * 2;
        const uint16_t *tile = base + (size_t)j * (BN * D);
        const uint32_t left = (uint32_t)a.Sk * (D * 2) - (uint32_t)j * tile_bytes;
        const tileattn_dma::u32x4s rs = tileattn_dma::buffer_rsrc(tile, left);
        const uint32_t lds0 = tileattn_dma::lds_addr(buf) + wave_u * 64 * 16;
        const uint32_t o0 = IS_V ? voff : koff;
        if ((j + 1) * BN <= a.Sk) {
#pragma unroll
            for (int i = 0; i < C::DMA_PER_THREAD; ++i)
                tileattn_dma::dma16_soff(lds0 + i * NT * 16, o0, i * NT * 16, rs);
        } else {
            const int last_row = a.Sk - 1 - j * BN;
            const int r0 = (int)(o0 / (2 * D));
#pragma unroll
            for (int i = 0; i < C::DMA_PER_THREAD; ++i) {
                const uint32_t o = r0 + i * RPS > last_row
                                       ? last_row * (2 * D) + o0 % (2 * D)
                                       : o0 + i * NT * 16;
                tileattn_dma::dma16(lds0 + i * NT * 16, o, rs);
            }
        }
    }

    __device__ __forceinline__ void dma_kv(size_t kv_base, int j, const unsigned char *stage) const
    {
        dma_tile<false>(a.K + kv_base, j, stage);
        dma_tile<true>(a.V + kv_base, j, stage + C::TILE_BYTES);
    }

    // S^T[key][query] of one tile (NKB blocks of QW keys, chains interleaved).
    // Each MFMA's K operand is read PF_S MFMAs ahead and scheduling barriers
    // keep that order (the compiler's own schedule kept one to three reads
    // in flight); the P V product below does the same with PF_V.
    __device__ __forceinline__ void scores(const unsigned char *kbuf, Acc (&s)[NKB]) const
    {
#pragma unroll
        for (int b = 0; b < NKB; ++b)
#pragma unroll
            for (int r = 0; r < AR; ++r)
                s[b][r] = 0.f;
        constexpr int N = KK * NKB;
        auto operand = [&](int i) -> bf16x8 {
            const int kk = i / NKB, b = i % NKB;
            const int row = QW * b + col;
            const int ch = (NG * kk + half) ^ C::kswz(row);
            return *(const bf16x8 *)(kbuf + row * (D * 2) + ch * 16);
        };
        bf16x8 buf[PF_S];
#pragma unroll
        for (int i = 0; i < PF_S; ++i)
            if (i < N)
                buf[i] = operand(i);
#pragma unroll
        for (int i = 0; i < N; ++i) {
            __builtin_amdgcn_sched_barrier(0);
            s[i % NKB] = mfma(buf[i % PF_S], qreg[i / NKB], s[i % NKB]);
            if (i + PF_S < N)
                buf[i % PF_S] = operand(i + PF_S);
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    // key (within the tile) of accumulator value r of block b
    __device__ __forceinline__ int key_of(int b, int r) const
    {
        return QW == 32 ? 32 * b + 8 * (r >> 2) + 4 * half + (r & 3) : 16 * b + 4 * half + r;
    }

    // Online softmax, first half: mask, row max, and (when some row's tile
    // max passes its level m_trig) raise the running max and rescale the
    // accumulator.
    template <bool MASKED>
    __device__ __forceinline__ void row_max(int j, Acc (&s)[NKB])
    {
        // lane holds keys j*BN + key_of(b, r) of query qi
        float mx = -INFINITY;
#pragma unroll
        for (int b = 0; b < NKB; ++b)
#pragma unroll
            for (int r = 0; r < AR; ++r) {
                if (MASKED) {
                    const int key = j * BN + key_of(b, r);
                    const bool ok = key < a.Sk && (!CAUSAL || key <= qi + off);
                    s[b][r] = ok ? s[b][r] : -INFINITY;
                }
                mx = fmaxf(mx, s[b][r]);
            }
        mx = max_halves(mx);
        if (QW == 16)
            mx = max_rows16(mx);
        const float m_tile = MASKED && mx == -INFINITY ? -INFINITY : mx * a.c;
        // raise the running max when some row passes its level (a
        // wave-uniform decision; every lane of the wave then rescales, by 1
        // where its own max did not move)
        if (__builtin_amdgcn_ballot_w64(m_tile > m_trig)) {
            // (the branch is wave-uniform: a lane whose row has seen no key
            // yet may have m_run = m_tile = -inf; its alpha is 1, not NaN)
            const float m_new = fmaxf(m_run, m_tile);
            const float alpha = m_new == -INFINITY
                                    ? 1.f
                                    : __builtin_amdgcn_exp2f(m_run - m_new);  // 0 if m_run = -inf
            m_run = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int r = 0; r < AR; ++r)
                    acc_o[db][r] *= alpha;
        }
    }

    // Online softmax, second half: weights exp2(c*s - m), row sum, bf16
    // weights, then O^T += V^T P^T
    template <bool MASKED>
    __device__ __forceinline__ void exp_pv(const Acc (&s)[NKB], const unsigned char *vbuf)
    {
        const float m_use = MASKED && m_run == -INFINITY ? 0.f : m_run;
        float rowsum = 0.f;
        uint32_t pk[NKB][AR / 2];
#pragma unroll
        for (int b = 0; b < NKB; ++b)
#pragma unroll
            for (int r = 0; r < AR; r += 2) {
                float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][r], a.c, -m_use));
                float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][r + 1], a.c, -m_use));
                if (MASKED) {
                    p0 = s[b][r] == -INFINITY ? 0.f : p0;
                    p1 = s[b][r + 1] == -INFINITY ? 0.f : p1;
                }
                rowsum += p0 + p1;
                pk[b][r >> 1] = pack_bf16(p0, p1);
            }
        l_run += rowsum;
        // the level for the next tile: m + min(8, max(0, log2(l / 4)));
        // l = 0 (no key seen yet) gives m itself
        m_trig = m_run + fminf(RESCALE_SLACK,
                               fmaxf(0.f, RAISE_SHARE_LOG2 + __builtin_amdgcn_logf(l_run)));

        // The A operand (V^T) comes from the row-major V tile through the
        // transpose read ds_read_b64_tr_b16: in each group of 16 lanes, lane
        // 4i + c reads dims d0 + 4c .. d0 + 4c + 3 of key row r0 + i, and lane
        // j of the group receives dim d0 + j of rows r0 .. r0 + 3, one dim
        // over 4 consecutive keys.
        const int sl = lane & 15;
        if constexpr (QW == 32) {
            // MFMA k-slot t of half h stands for key 16ks + 4h + t (t < 4) or
            // 16ks + 8 + 4h + t-4, matching where the accumulator layout left P
            const int gq = lane >> 4;
            constexpr int N = (BN / 16) * DB;
            auto operand = [&](int i) -> bf16x8 {
                const int ks = i / DB, db = i % DB;
                const int row0 = 16 * ks + 4 * half + (sl >> 2);
                const int d = 32 * db + 16 * (gq & 1) + 4 * (sl & 3);
                return v_operand(vbuf, row0, row0 + 8, d);
            };
            bf16x8 buf[PF_V];
#pragma unroll
            for (int i = 0; i < PF_V; ++i)
                if (i < N)
                    buf[i] = operand(i);
#pragma unroll
            for (int i = 0; i < N; ++i) {
                __builtin_amdgcn_sched_barrier(0);
                const int ks = i / DB, db = i % DB;
                const int b = ks >> 1, rb = (ks & 1) * 4;
                const u32x4 bw = {pk[b][rb], pk[b][rb + 1], pk[b][rb + 2], pk[b][rb + 3]};
                acc_o[db] = mfma(buf[i % PF_V], __builtin_bit_cast(bf16x8, bw), acc_o[db]);
                if (i + PF_V < N)
                    buf[i % PF_V] = operand(i + PF_V);
            }
            __builtin_amdgcn_sched_barrier(0);
        } else {
            // MFMA k-slot t of quarter g stands for key 32ks + 4g + t (t < 4)
            // or 32ks + 16 + 4g + t-4: blocks 2ks and 2ks+1 of the scores
            constexpr int N = (BN / 32) * DB;
            auto operand = [&](int i) -> bf16x8 {
                const int ks = i / DB, db = i % DB;
                const int row0 = 32 * ks + 4 * half + (sl >> 2);
                return v_operand(vbuf, row0, row0 + 16, 16 * db + 4 * (sl & 3));
            };
            bf16x8 buf[PF_V];
#pragma unroll
            for (int i = 0; i < PF_V; ++i)
                if (i < N)
                    buf[i] = operand(i);
#pragma unroll
            for (int i = 0; i < N; ++i) {
                __builtin_amdgcn_sched_barrier(0);
                const int ks = i / DB, db = i % DB;
                const u32x4 bw = {pk[2 * ks][0], pk[2 * ks][1], pk[2 * ks + 1][0],
                                  pk[2 * ks + 1][1]};
                acc_o[db] = mfma(buf[i % PF_V], __builtin_bit_cast(bf16x8, bw), acc_o[db]);
                if (i + PF_V < N)
                    buf[i % PF_V] = operand(i + PF_V);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    // 4 dims from d of V rows row0 (k-slots 0..3) and row1 (k-slots 4..7),
    // transposed across lanes (see above)
    __device__ __forceinline__ bf16x8 v_operand(const unsigned char *vbuf, int row0, int row1,
                                                int d) const
    {
        const int byte_in = (2 * d) & 15;
        const unsigned char *p0 = vbuf + row0 * (D * 2) + ((d >> 3) ^ C::vswz(row0)) * 16 + byte_in;
        const unsigned char *p1 = vbuf + row1 * (D * 2) + ((d >> 3) ^ C::vswz(row1)) * 16 + byte_in;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p0);
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p1);
        const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
        const u32x4 aw = {l2[0], l2[1], h2[0], h2[1]};
        return __builtin_bit_cast(bf16x8, aw);
    }

    // wave w sees tile j unless every key in it is beyond its last query
    __device__ __forceinline__ bool active(int j) const
    {
        return wave_has_rows && (!CAUSAL || j * BN <= q_last_wave + off);
    }

    // Tile j of the current item from the stage at `sc` (K tile, then V
    // tile).  First the DMA of the next tile of the workgroup's stream goes
    // into the other stage `sn`: tile j+1 of this item, or on its last tile
    // the first tile of the next item.  MASKED = false: the tile is fully
    // visible to every real query of the item (a wave holding only padding
    // rows past Sq computes on it and never stores).  MASKED = true: waves
    // skip the tile if they cannot see any of it.  Every thread takes part
    // in the DMA and the barrier.
    template <bool MASKED>
    __device__ __forceinline__ void tile(int j, const unsigned char *sc, const unsigned char *sn)
    {
        const bool last = j + 1 == cur.j_hi;
        if (!last || has_next)
            dma_kv(last ? nxt.kv_base : cur.kv_base, last ? nxt.j_lo : j + 1, sn);
        const bool act = !MASKED || active(j);   // wave-uniform
        Acc s[NKB];
        if (act)
            scores(sc, s);
        if (last && has_next) {
            // the next item's Q, once this tile's score MFMAs (the last
            // readers of Q) are issued
            __builtin_amdgcn_sched_barrier(0);
            load_q(nxt);
        }
        if (act) {
            row_max<MASKED>(j, s);
            exp_pv<MASKED>(s, sc + C::TILE_BYTES);
        }
        tileattn_dma::wait_vmcnt<0>();
        __syncthreads();
    }

    // Epilogue of the current item: normalise, store O rows (fp32, or bf16
    // rounded to nearest even) and LSE.  A row that saw no key of its split
    // (only possible with key splits) stores the empty partial result:
    // O = 0, LSE = -inf.
    //   The rows go through LDS so that every store instruction writes whole
    // rows (lane (col, half) holds runs of 4 consecutive dims of row col:
    // written directly, each instruction would write pieces of 16 or 8
    // bytes).  The staging area is the stage of the item's last tile, which
    // every wave has left behind at that tile's barrier (the other stage
    // holds the next item's first tile, in flight), or all of LDS in a grid
    // of one workgroup per item; each wave
    // stages RP of its QW rows at a time in its own quarter, 16-byte chunk q
    // of staged row r at q ^ (r % RCH), and reads back only what it wrote
    // itself (a wave's LDS accesses complete in order).  A barrier then
    // keeps the next item's DMA into this stage behind every wave's reads;
    // the stores complete in the background, during the next item's first
    // tile.
    template <bool WHOLE_LDS>
    __device__ __forceinline__ void epilogue(unsigned char *stage)
    {
        const float l = QW == 32 ? sum_halves(l_run) : sum_rows16(sum_halves(l_run));
        const bool empty = !(l > 0.f);
        const float inv = empty ? 0.f : 1.f / l;
        constexpr int EB = OBF16 ? 2 : 4;               // bytes per output element
        constexpr int RCH = D * EB / 16;                // 16-byte chunks per row
        constexpr int RPI = 64 / RCH;                   // rows per read instruction
        // each wave's quarter of the staging area: of the last tile's stage,
        // or (WHOLE_LDS: one item per workgroup, no DMA in flight) of all of LDS
        constexpr int QB = (WHOLE_LDS ? 4 : 2) * C::TILE_BYTES / 4;
        constexpr int RP = QB / (D * EB) < QW ? QB / (D * EB) : QW;  // rows per pass
        constexpr int NP = QW / RP;                     // passes
        constexpr int NI = RP / RPI;                    // reads per pass
        static_assert(RP % RPI == 0 && QW % RP == 0, "staging shape");
        unsigned char *const stg = stage + wave * QB;
        // O elements of this item's first row (the split's partial results
        // start o_split elements apart; bf16 O is never split)
        const size_t obase = (OBF16 ? 0 : (size_t)cur.split * a.o_split) + cur.row0 * D;
        // the lane coordinates as opaque values here, so that the staging
        // addresses are computed here, once per item, and not kept in
        // registers (or spilled) across the tile loop
        int col = this->col, half = this->half, lane = this->lane;
        asm volatile("" : "+v"(col), "+v"(half), "+v"(lane));
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            if (col / RP == p) {
                const int r = col % RP;
                // accumulator values 4g .. 4g+3 of block db: dims
                // QW db + (QW == 32 ? 8 g + 4 half : 4 half) .. +3
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int g = 0; g < AR / 4; ++g) {
                        const int dim = QW * db + (QW == 32 ? 8 * g : 0) + 4 * half;
                        const int byte = dim * EB;   // within the row
                        unsigned char *pp =
                            stg + r * (D * EB) + (((byte >> 4) ^ (r & (RCH - 1))) * 16) + (byte & 15);
                        const float x0 = acc_o[db][4 * g + 0] * inv, x1 = acc_o[db][4 * g + 1] * inv;
                        const float x2 = acc_o[db][4 * g + 2] * inv, x3 = acc_o[db][4 * g + 3] * inv;
                        if (OBF16)
                            *(u32x2 *)pp = u32x2{pack_bf16(x0, x1), pack_bf16(x2, x3)};
                        else
                            *(float4 *)pp = float4{x0, x1, x2, x3};
                    }
            }
            if (p == 0) {
                // Q has landed before any store is issued: the compiler's own
                // wait for Q, at the next item's first scores, then finds no
                // load of its own pending and cannot end up waiting for that
                // item's tile DMA, which it does not track (unconditional, so
                // that it covers every path from the load)
                tileattn_dma::wait_vmcnt<0>();
            }
#pragma unroll
            for (int it = 0; it < NI; ++it) {
                const int r = it * RPI + lane / RCH, q = lane % RCH;
                const u32x4 v = *(const u32x4 *)(stg + r * (D * EB) + ((q ^ (r & (RCH - 1))) * 16));
                const int qr = cur.q0 + wave * QW + p * RP + r;
                if (qr < a.Sq) {
                    if (OBF16)
                        *(u32x4 *)((uint16_t *)a.O + obase + (size_t)qr * D + 8 * q) = v;
                    else
                        *(u32x4 *)((float *)a.O + obase + (size_t)qr * D + 4 * q) = v;
                }
            }
        }
        if (qi < a.Sq && half == 0)
            a.LSE[(size_t)cur.split * a.l_split + cur.row0 + qi] =
                empty ? -INFINITY : (m_run + log2f(l)) * LN2;
        if (has_next) {
            // every wave's staging reads complete before any wave's next DMA
            // into this stage (the stores need not have completed)
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
            __builtin_amdgcn_s_barrier();
        }
    }

    // The key tiles of the current item, the first in stage `st` (its DMA
    // already waited for): those before j_fast in one loop, unrolled by two
    // so that both stage addresses are fixed for the item, the masked ones
    // in another.  Returns the stage holding the next item's first tile.
    __device__ __forceinline__ int run_item(unsigned char *lds, int st)
    {
        constexpr int SB = 2 * C::TILE_BYTES;   // bytes per stage
        unsigned char *sa = lds + st * SB, *sb = lds + (st ^ 1) * SB;
        int j = cur.j_lo;
        for (; j + 1 < cur.j_fast; j += 2) {
            tile<false>(j, sa, sb);
            tile<false>(j + 1, sb, sa);
        }
        if (j < cur.j_fast) {
            tile<false>(j, sa, sb);
            unsigned char *const t = sa;
            sa = sb;
            sb = t;
            ++j;
        }
        for (; j < cur.j_hi; ++j) {
            tile<true>(j, sa, sb);
            unsigned char *const t = sa;
            sa = sb;
            sb = t;
        }
        if (PERSIST)
            epilogue<false>(sb);
        else
            epilogue<true>(lds);
        return sa == lds ? 0 : 1;
    }

    // An item whose key split holds no visible key (key splits only, one
    // item per workgroup): the empty partial result, LSE = -inf and O = 0,
    // which the combine step weights by zero.
    __device__ void empty_result(int tid) const
    {
        const int r = cur.q0 + tid / 2;
        if (tid < 2 * BMQ && r < a.Sq) {
            float *op = (float *)a.O + (size_t)cur.split * a.o_split + (cur.row0 + r) * D;
#pragma unroll
            for (int d = (tid & 1) * (D / 2); d < (tid & 1) * (D / 2) + D / 2; d += 4)
                *(float4 *)(op + d) = float4{0.f, 0.f, 0.f, 0.f};
            if ((tid & 1) == 0)
                a.LSE[(size_t)cur.split * a.l_split + cur.row0 + r] = -INFINITY;
        }
    }
};

// A workgroup computes its items one after another as one stream of key
// tiles: the DMA of the next item's first tile and the load of its Q overlap
// the current item's last tile, and the current item's O stores overlap the
// next item's first tile.  The grid is either one workgroup per item or two
// resident workgroups per CU looping over the items (persistent).  QW = 16
// workgroups use half the registers, so up to four fit a CU where LDS
// allows (D = 64).
template <int D, int QW, bool CAUSAL, bool OBF16, bool PERSIST>
__global__ __launch_bounds__(NT, QW == 16 && D == 64 ? 4 : 2) void attn_fwd_kernel(Args args)
{
    using C = Cfg<D>;
    // two stages, each a K tile then a V tile
    __shared__ __attribute__((aligned(16))) unsigned char lds[4 * C::TILE_BYTES];

    Kernel<D, QW, CAUSAL, OBF16, PERSIST> k(args);
    const Args &a = args;
    const int tid = threadIdx.x;
    k.wave = tid >> 6;
    k.lane = tid & 63;
    k.col = k.lane % QW;
    k.half = k.lane / QW;
    k.off = a.Sk - a.Sq;

    int L = PERSIST ? persistent_item(a, blockIdx.x, gridDim.x, 0) : static_item(a, blockIdx.x);
    if (L < 0)
        return;
    k.cur = k.describe(L);
    if (k.cur.j_lo >= k.cur.j_hi) {
        // (key splits only: such a grid has one workgroup per item)
        k.empty_result(tid);
        return;
    }
    k.init_dma();
    k.set_rows();
    k.load_q(k.cur);
    // prologue: the first tile in stage 0
    k.dma_kv(k.cur.kv_base, k.cur.j_lo, lds);
    tileattn_dma::wait_vmcnt<0>();
    __syncthreads();

    int st = 0;
    for (int r = 1;; ++r) {
        L = PERSIST ? persistent_item(a, blockIdx.x, gridDim.x, r) : -1;
        k.has_next = L >= 0;
        if (k.has_next)
            k.nxt = k.describe(L);
        k.reset_state();
        st = k.run_item(lds, st);
        if (!k.has_next)
            break;
        k.cur = k.nxt;
        k.set_rows();
    }
}

// One workgroup per item when `grid` covers the items, else the persistent
// kernel (no key splits then); 64-query workgroups (16 rows per wave) for
// small grids, one workgroup per item.
template <int D, bool CAUSAL, bool OBF16>
hipError_t launch(const Args &a, int grid, bool small, hipStream_t stream)
{
    if (small)
        hipLaunchKernelGGL((attn_fwd_kernel<D, 16, CAUSAL, OBF16, false>), dim3(grid), dim3(NT),
                           0, stream, a);
    else if (grid < a.n_items)
        hipLaunchKernelGGL((attn_fwd_kernel<D, 32, CAUSAL, OBF16, true>), dim3(grid), dim3(NT), 0,
                           stream, a);
    else
        hipLaunchKernelGGL((attn_fwd_kernel<D, 32, CAUSAL, OBF16, false>), dim3(grid), dim3(NT), 0,
                           stream, a);
    return hipGetLastError();
}

// Workgroups of the attention kernel resident at once per CU (its LDS, four
// tile buffers, and registers allow two).  A causal grid with more items
// than resident workgroups is launched persistent: this many workgroups per
// CU, each looping over its share of the items (measured on one MI355X:
// grouped-query S=4096 +6 %, B=1 H=32 S=4096 +10 %, S=8192 unchanged).
// Non-causal items all cost the same, and there the grid of one workgroup
// per item measured 4-5 % faster than the persistent one (B=8 H=32 S=2048).
#ifndef TA_RESIDENT_PER_CU
#define TA_RESIDENT_PER_CU 2
#endif
constexpr int MAX_DEVICES = 64;
std::atomic<int> cu_count[MAX_DEVICES];

// CUs of the current device (0 if the runtime cannot tell), looked up once
// per device.
int current_cu_count()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES)
        return 0;
    int n = cu_count[dev].load(std::memory_order_relaxed);
    if (n <= 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n <= 0)
            return 0;
        cu_count[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Grid size for n_items work items on a device with n_cu CUs (one
// workgroup per item unless the persistent grid is smaller; a multiple of
// the XCD count).
int grid_size(int n_items, int n_split, bool causal, int n_cu)
{
    if (TA_RESIDENT_PER_CU < 1 || n_split != 1 || !causal)
        return n_items;
    const int g = (TA_RESIDENT_PER_CU * n_cu) / NXCD * NXCD;
    return g >= NXCD && n_items > g ? g : n_items;
}

// Grids of 128-query tiles that would leave at least half of the CUs
// without a workgroup run as 64-query workgroups (16 query rows per wave)
// instead: twice the workgroups, each wave's chain of key tiles half as long
// in MFMA and softmax work (measured on one MI355X: B=1 H=32 S=512 causal
// 134 -> 170 and non-causal 288 -> 340 TFLOP/s).  So do causal grids of at
// most one 128-query workgroup per CU whose query tiles differ in cost by
// more than a factor of two (Sk - Sq < Sq): their heavy and light 64-query
// tiles pair up on the CUs (B=1 H=32 S=1024 causal 324 -> 370).  Where the
// costs are even (non-causal, or a short query chunk against a long key
// range) a 64-query grid with two workgroups per CU measured 7-9 % slower
// than the 128-query grid (its waves read each K/V tile from LDS for half
// as many queries).
#ifndef TA_SMALL_TILES
#define TA_SMALL_TILES 1
#endif

bool overlaps(const void *p, size_t pn, const void *q, size_t qn)
{
    const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + qn && b < a + pn;
}

bool misaligned(const void *p) { return ((uintptr_t)p & 15u) != 0; }

// Integer tile schedule; must agree with the kernel's own loop bounds.
void schedule(int Sq, int Sk, int causal, int qt, int *n_kv, int *first_masked)
{
    const int n_all = (Sk + BN - 1) / BN;
    int n = n_all;
    int fm = (Sk % BN) ? n_all - 1 : n_all;
    if (causal) {
        const int q0 = qt * BM;
        const int q_last = (q0 + BM < Sq ? q0 + BM : Sq) - 1;
        const int off = Sk - Sq;
        const int lim = (q_last + off) / BN + 1;
        n = lim < n_all ? lim : n_all;
        int cm = (q0 + off + 1) / BN;
        if (cm < 0)
            cm = 0;
        fm = fm < cm ? fm : cm;
        fm = fm < n ? fm : n;
    }
    *n_kv = n;
    *first_masked = fm;
}

constexpr int MAX_SPLITS = 128;
// split heuristic: aim for two resident workgroups per CU (256 CUs), with at
// least 32 key tiles (2048 keys) per split, so that the work of a split
// outweighs the second launch and the partial-result traffic of the merge
constexpr int64_t SPLIT_TARGET_WG = 512;
constexpr int SPLIT_MIN_TILES = 32;

// Key tiles per split and the number of splits actually launched for a
// requested split count (trailing splits that would start past the last key
// tile are dropped).
void split_shape(int Sk, int num_splits, int *split_tiles, int *n_split)
{
    const int n_kv_all = (Sk + BN - 1) / BN;
    const int per = (n_kv_all + num_splits - 1) / num_splits;
    *split_tiles = per;
    *n_split = (n_kv_all + per - 1) / per;
}

size_t split_workspace_bytes(int B, int Hq, int Sq, int D, int num_splits)
{
    const size_t rows = (size_t)B * Hq * Sq;
    return (size_t)num_splits * rows * (size_t)(D + 1) * 4;
}

// Validation and launch shared by every entry point.  num_splits == 1 runs
// one kernel writing O and LSE; num_splits > 1 writes per-split partial
// results into the workspace and merges them with combine_kernel.
ta_status attn_fwd_any(const void *Q, const void *K, const void *V, void *O, bool o_bf16,
                       float *LSE, int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                       float scale, int num_splits, void *ws, size_t ws_bytes, void *stream,
                       bool validate_only = false)
{
    if (!Q || !K || !V || !O || !LSE)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Sk < 1 || D < 1)
        return TA_ERR_INVALID_SHAPE;
    if (Hq % Hkv != 0 || (causal && Sq > Sk))
        return TA_ERR_INVALID_SHAPE;
    if (num_splits < 1 || num_splits > MAX_SPLITS)
        return TA_ERR_INVALID_SHAPE;
    if (D != 64 && D != 128)
        return TA_ERR_UNSUPPORTED;
    int split_tiles, n_split;
    split_shape(Sk, num_splits, &split_tiles, &n_split);
    // 32-bit in-kernel offsets are used within one (batch, head) slice only;
    // the grid itself must fit a 32-bit workgroup count
    const int64_t n_qt = ((int64_t)Sq + BM - 1) / BM;
    const int64_t n_items = (int64_t)B * Hq * n_qt * n_split;
    const int64_t n_rows = (int64_t)B * Hq * Sq;
    if ((int64_t)Sq * D >= (1ll << 31) || (int64_t)Sk * D >= (1ll << 31) ||
        n_items >= (1ll << 31) || n_rows >= (1ll << 31))
        return TA_ERR_INVALID_SHAPE;
    if (misaligned(Q) || misaligned(K) || misaligned(V) || misaligned(O) || misaligned(LSE))
        return TA_ERR_MISALIGNED;
    if (!(scale >= 0.f) || !isfinite(scale))
        return TA_ERR_INVALID_SCALE;
    const size_t nq = (size_t)B * Hq * Sq * D, nkv = (size_t)B * Hkv * Sk * D;
    const size_t nl = (size_t)n_rows;
    const size_t o_bytes = nq * (o_bf16 ? 2 : 4), l_bytes = nl * 4;
    if (overlaps(O, o_bytes, Q, nq * 2) || overlaps(O, o_bytes, K, nkv * 2) ||
        overlaps(O, o_bytes, V, nkv * 2) || overlaps(LSE, l_bytes, Q, nq * 2) ||
        overlaps(LSE, l_bytes, K, nkv * 2) || overlaps(LSE, l_bytes, V, nkv * 2) ||
        overlaps(O, o_bytes, LSE, l_bytes))
        return TA_ERR_ALIASING;
    const size_t need = n_split > 1 ? split_workspace_bytes(B, Hq, Sq, D, n_split) : 0;
    if (validate_only)
        return TA_OK;
    if (n_split > 1) {
        if (!ws || ws_bytes < need)
            return TA_ERR_WORKSPACE;
        if (misaligned(ws))
            return TA_ERR_MISALIGNED;
        if (overlaps(ws, need, Q, nq * 2) || overlaps(ws, need, K, nkv * 2) ||
            overlaps(ws, need, V, nkv * 2) || overlaps(ws, need, O, o_bytes) ||
            overlaps(ws, need, LSE, l_bytes))
            return TA_ERR_ALIASING;
    }

    Args a;
    a.Q = (const uint16_t *)Q;
    a.K = (const uint16_t *)K;
    a.V = (const uint16_t *)V;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.Sq = Sq;
    a.Sk = Sk;
    a.group = Hq / Hkv;
    a.n_qt = (int)n_qt;
    a.n_split = n_split;
    a.split_tiles = split_tiles;
    a.n_items = (int)n_items;
    a.c = scale * LOG2E;
    // split partial results: O then LSE of every split (no workspace for one split)
    float *Op = (float *)ws;
    float *Lp = n_split > 1 ? Op + (size_t)n_split * nq : nullptr;
    if (n_split > 1) {
        a.O = Op;
        a.LSE = Lp;
        a.o_split = nq;
        a.l_split = nl;
    } else {
        a.O = O;
        a.LSE = LSE;
        a.o_split = 0;
        a.l_split = 0;
    }

    hipStream_t s = (hipStream_t)stream;
    const int n_cu = current_cu_count();
    const bool small = TA_SMALL_TILES && n_split == 1 && n_cu > 0 &&
                       (2 * n_items <= (int64_t)n_cu ||
                        (causal && Sk - Sq < Sq && n_items <= (int64_t)n_cu));
    if (small) {
        a.n_qt = (Sq + BM_SMALL - 1) / BM_SMALL;
        a.n_items = B * Hq * a.n_qt;
    }
    a.cu_per_xcd = n_cu % NXCD == 0 ? n_cu / NXCD : 0;
    const int grid = small ? a.n_items : grid_size(a.n_items, n_split, causal != 0, n_cu);
    hipError_t e;
    const bool kb = o_bf16 && n_split == 1;   // the attention kernel writes bf16 O itself
    if (kb) {
        if (D == 64)
            e = causal ? launch<64, true, true>(a, grid, small, s)
                       : launch<64, false, true>(a, grid, small, s);
        else
            e = causal ? launch<128, true, true>(a, grid, small, s)
                       : launch<128, false, true>(a, grid, small, s);
    } else {
        if (D == 64)
            e = causal ? launch<64, true, false>(a, grid, small, s)
                       : launch<64, false, false>(a, grid, small, s);
        else
            e = causal ? launch<128, true, false>(a, grid, small, s)
                       : launch<128, false, false>(a, grid, small, s);
    }
    if (e == hipSuccess && n_split > 1) {
        const int nr = (int)n_rows;
        if (D == 64)
            e = o_bf16 ? tileattn_detail::launch_combine<64, true>(Op, Lp, O, LSE, nr, n_split, nq, nl, s)
                       : tileattn_detail::launch_combine<64, false>(Op, Lp, O, LSE, nr, n_split, nq, nl, s);
        else
            e = o_bf16 ? tileattn_detail::launch_combine<128, true>(Op, Lp, O, LSE, nr, n_split, nq, nl, s)
                       : tileattn_detail::launch_combine<128, false>(Op, Lp, O, LSE, nr, n_split, nq, nl, s);
    }
    return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH;
}

// Per-device address of `tileattn_split_scratch` (declared below, outside
// this namespace), looked up once per device with that device current.
std::atomic<void *> scratch_addr[MAX_DEVICES];

}  // namespace

// Partial results of attn_fwd_split_noalloc: a file-scope device array
// instead of a caller workspace, for callers that cannot allocate.  Each GPU
// the library runs on holds its own copy until the process ends.  In host
// code the name stands for a host-side shadow, never a device address: host
// code uses the address hipGetSymbolAddress returns for the current device.
// The array has external linkage: the runtime finds it by name among the
// global symbols of the device code object, and a `static` array is a local
// symbol there (the lookup then aborts the process).
__device__ __align__(256) unsigned char tileattn_split_scratch[TA_SPLIT_SCRATCH_BYTES];

namespace {

// The device address of `tileattn_split_scratch` on the current device
// (TA_ERR_LAUNCH if the runtime cannot report the device or the address).
ta_status scratch_on_current_device(void **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES)
        return TA_ERR_LAUNCH;
    void *p = scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(tileattn_split_scratch)) != hipSuccess || !p)
            return TA_ERR_LAUNCH;
        scratch_addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return TA_OK;
}

}  // namespace

extern "C" {

ta_status attn_fwd(const void *Q, const void *K, const void *V, float *O, float *LSE, int B,
                   int Hq, int Hkv, int Sq, int Sk, int D, int causal, float scale, void *stream)
{
    return attn_fwd_any(Q, K, V, O, false, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, 1, nullptr,
                        0, stream);
}

ta_status attn_fwd_bf16out(const void *Q, const void *K, const void *V, void *O, float *LSE,
                           int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                           float scale, void *stream)
{
    return attn_fwd_any(Q, K, V, O, true, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, 1, nullptr,
                        0, stream);
}

ta_status attn_fwd_split(const void *Q, const void *K, const void *V, void *O, int o_bf16,
                         float *LSE, int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                         float scale, int num_splits, void *workspace, size_t workspace_bytes,
                         void *stream)
{
    return attn_fwd_any(Q, K, V, O, o_bf16 != 0, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale,
                        num_splits, workspace, workspace_bytes, stream);
}

ta_status attn_fwd_split_noalloc(const void *Q, const void *K, const void *V, void *O,
                                 int o_bf16, float *LSE, int B, int Hq, int Hkv, int Sq, int Sk,
                                 int D, int causal, float scale, int num_splits, void *stream)
{
    // every argument check first, then the size check, then HIP calls
    ta_status st = attn_fwd_any(Q, K, V, O, o_bf16 != 0, LSE, B, Hq, Hkv, Sq, Sk, D, causal,
                                scale, num_splits, nullptr, 0, stream, true);
    if (st != TA_OK)
        return st;
    int split_tiles, n_split;
    split_shape(Sk, num_splits, &split_tiles, &n_split);
    if (n_split == 1)
        return attn_fwd_any(Q, K, V, O, o_bf16 != 0, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale,
                            1, nullptr, 0, stream);
    if (split_workspace_bytes(B, Hq, Sq, D, n_split) > TA_SPLIT_SCRATCH_BYTES)
        return TA_ERR_SCRATCH;
    void *ws = nullptr;
    st = scratch_on_current_device(&ws);
    if (st != TA_OK)
        return st;
    return attn_fwd_any(Q, K, V, O, o_bf16 != 0, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale,
                        num_splits, ws, TA_SPLIT_SCRATCH_BYTES, stream);
}

ta_status ta_split_workspace_bytes(int B, int Hq, int Sq, int D, int num_splits, size_t *bytes)
{
    if (!bytes)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || Hq < 1 || Sq < 1 || num_splits < 1 || num_splits > MAX_SPLITS)
        return TA_ERR_INVALID_SHAPE;
    if (D != 64 && D != 128)
        return TA_ERR_UNSUPPORTED;
    *bytes = num_splits > 1 ? split_workspace_bytes(B, Hq, Sq, D, num_splits) : 0;
    return TA_OK;
}

ta_status ta_split_heuristic(int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                             int *num_splits)
{
    if (!num_splits)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Sk < 1 || Hq % Hkv != 0 || (causal && Sq > Sk))
        return TA_ERR_INVALID_SHAPE;
    if (D != 64 && D != 128)
        return TA_ERR_UNSUPPORTED;
    const int64_t n_wg = (int64_t)B * Hq * (((int64_t)Sq + BM - 1) / BM);
    const int n_kv_all = (Sk + BN - 1) / BN;
    int n = 1;
    if (n_wg < SPLIT_TARGET_WG) {
        n = (int)((SPLIT_TARGET_WG + n_wg - 1) / n_wg);
        n = n < n_kv_all / SPLIT_MIN_TILES ? n : n_kv_all / SPLIT_MIN_TILES;
        n = n < MAX_SPLITS ? n : MAX_SPLITS;
        n = n > 1 ? n : 1;
    }
    *num_splits = n;
    return TA_OK;
}

ta_status ta_schedule(int Sq, int Sk, int D, int causal, int q_tile, int *n_kv_tiles,
                      int *first_masked)
{
    if (!n_kv_tiles || !first_masked)
        return TA_ERR_NULL_POINTER;
    if (D != 64 && D != 128)
        return TA_ERR_UNSUPPORTED;
    if (Sq < 1 || Sk < 1 || (causal && Sq > Sk))
        return TA_ERR_INVALID_SHAPE;
    if (q_tile < 0 || (int64_t)q_tile * BM >= Sq)
        return TA_ERR_INVALID_SHAPE;
    schedule(Sq, Sk, causal, q_tile, n_kv_tiles, first_masked);
    return TA_OK;
}

ta_status ta_tile_shape(int D, int *bm, int *bn)
{
    if (!bm || !bn)
        return TA_ERR_NULL_POINTER;
    if (D != 64 && D != 128)
        return TA_ERR_UNSUPPORTED;
    *bm = BM;
    *bn = BN;
    return TA_OK;
}

const char *ta_status_string(ta_status s)
{
    switch (s) {
    case TA_OK: return "ok";
    case TA_ERR_NULL_POINTER: return "null pointer";
    case TA_ERR_INVALID_SHAPE: return "invalid shape";
    case TA_ERR_UNSUPPORTED: return "unsupported head dim (D must be 64 or 128)";
    case TA_ERR_MISALIGNED: return "pointer not 16-byte aligned";
    case TA_ERR_INVALID_SCALE: return "scale must be finite and >= 0";
    case TA_ERR_ALIASING: return "output overlaps an input or the other output";
    case TA_ERR_LAUNCH: return "HIP launch error";
    case TA_ERR_WORKSPACE: return "split workspace missing or too small";
    case TA_ERR_SCRATCH: return "partial results exceed the static split scratch";
    }
    return "unknown status";
}

int ta_version(void) { return 400; }

}  // extern "C"
