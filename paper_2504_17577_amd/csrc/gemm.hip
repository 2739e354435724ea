// bf16 matrix multiplication C = A B for gfx950 (MI355X): the kernel beneath
// the paper's Matmul listing (appendix "Matrix Multiplication (Matmul)":
// tiles of A [M, K] and B [K, N], row-major, copied to shared memory per
// K-step and multiplied into a register tile of C).  The design is this
// library's own for CDNA4:
//
//  * One workgroup of eight wave64s computes a BM x BN tile of C (256 x 256,
//    or 128 x 128 when the grid of large tiles would not fill the GPU); the
//    waves form a 2 x 4 grid, each owning (BM/2) x (BN/4) as 16 x 16 blocks
//    of v_mfma_f32_16x16x32_bf16 accumulators (fp32; 32 x 32 blocks of
//    v_mfma_f32_32x32x16_bf16 where four wave groups split each K step, see
//    below).  Under the board's power limit the 16 x 16 x 32 form sustains
//    a higher clock for the same work (random data, MFMAs alone: 2.15
//    against 1.84 GHz, 2.18-2.26 against 1.72 PFLOP/s).  Two waves share each
//    SIMD, so one's matrix-core work covers the other's LDS reads and
//    barrier waits.  Four waves of 128 x 128 each read a third less from LDS
//    per flop and run at a ~6 % higher clock under the board's power limit,
//    but with one wave per SIMD their matrix cores idle at every barrier and
//    operand wait: measured 1-3 % slower at 8192^3 and 4096 x 8192 x 8192.
//    128 x 128 tiles instead split every K step over two groups of four
//    waves (1 x 4 each) or, with one workgroup per CU, four groups of two
//    (1 x 2 each), each group covering the whole tile for its share of the
//    step: fewer operand reads per flop; the groups' sums meet in LDS.
//  * K advances in steps of 64.  The A tile [BM][64] and the B tile [64][BN]
//    go global -> LDS by DMA (buffer_load_dwordx4 ... lds, issued as inline
//    assembly and waited for explicitly), double-buffered: the DMA of step
//    k+1 runs under the MFMAs of step k.  With one workgroup per CU (small
//    grids of 128 x 128 tiles) a ring of four stages keeps three steps in
//    flight instead.
//  * A operands (16 or 32 rows x 8 consecutive k per lane) are ds_read_b128
//    from the A tile, 16-byte chunk c of row r stored at c ^ ((r >> 1) & 7).
//    B operands (8 consecutive k of one column per lane) come from the
//    row-major B tile through the transpose read ds_read_b64_tr_b16, chunk c
//    of row r stored at c ^ (2 (r & 3) + 8 ((r >> 3) & 1)) for 16 x 16
//    blocks (a half wave reads eight rows of 32 bytes) or c ^ 4 (r & 3) for
//    32 x 32 ones (four rows of 64 bytes).  The swizzles keep the operand
//    reads bank-conflict free.
//  * The grid maps workgroups so that each XCD gets a contiguous range of
//    tiles, taken in groups of four tile rows (column by column inside a
//    group), so the tiles resident on one XCD form a 4 x 8 block that shares
//    its A and B panels in that XCD's L2 (row-major order re-read each B
//    panel once per tile row: 4.4 GB of L2 misses per 8192^3 product).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tileattn.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int BK = 64;       // K per stage
constexpr int NT = 512;      // threads per workgroup (8 waves)
constexpr int NXCD = 8;
constexpr int GROUP_M = 4;   // tile rows per group of the grid order
[[maybe_unused]] constexpr int BUF_RSRC_WORD3 = 0x00020000;

struct GArgs {
    const uint16_t *A, *B;
    void *C;
    int M, N, K;
    int tiles_n;     // N / BN
    int n_wg;
};

[[maybe_unused]] __device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

[[maybe_unused]] __device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// The tile DMA is inline assembly, untracked by the compiler (it would
// otherwise drain the loads in flight before every LDS read, unable to tell
// which buffer they write); the loop waits for it with vmcnt(0).
__device__ __forceinline__ void wait_dma_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// wait until at most N of this thread's tile loads are outstanding (N < 16)
template <int N>
__device__ __forceinline__ void wait_dma_upto() { __builtin_amdgcn_s_waitcnt(0x0F70 | N); }

typedef uint32_t u32x4s __attribute__((ext_vector_type(4)));

// raw buffer resource (stride 0, 32-bit format, range-checked) in SGPRs
__device__ __forceinline__ u32x4s buffer_rsrc(const void *base, uint32_t bytes)
{
    const uint64_t a = (uint64_t)(uintptr_t)base;
    return u32x4s{(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a),
                  (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xFFFFu),
                  (uint32_t)__builtin_amdgcn_readfirstlane(bytes), (uint32_t)BUF_RSRC_WORD3};
}

// lane l's 16 bytes at byte `voff` of the buffer land at LDS `lds` + 16 l
// (`lds` wave-uniform, passed in M0: the compiler sets M0 for the statement)
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

__device__ __forceinline__ int a_swz(int r) { return (r >> 1) & 7; }
// B swizzle for the transpose reads of MF x MF blocks: MF = 32 reads four
// rows of 64 bytes per half wave, MF = 16 eight rows (4gq .. +3 of two lane
// groups, 8 apart) of 32 bytes, whose chunk pairs it keeps apart
template <int MF>
__device__ __forceinline__ int b_swz(int r)
{
    return MF == 32 ? 4 * (r & 3) : 2 * (r & 3) + 8 * ((r >> 3) & 1);
}

// KS = 1: the eight waves tile C as 2 x 4.  KS = 2 or 4: KS groups of 8 / KS
// waves, each group tiling C as 1 x (8 / KS) for its share of every K step
// (a wave then reads less of the tiles per flop, most of all of B through
// the transpose read); the groups' sums are added in LDS at the end.
template <int BM, int BN, int KS, int MF>
struct Cfg {
    static constexpr int WPG = 8 / KS;                               // waves per group
    static constexpr int WM = KS == 1 ? BM / 2 : BM, WN = KS == 1 ? BN / 4 : BN / WPG;
    static constexpr int FM = WM / MF, FN = WN / MF;      // MF x MF blocks per wave
    static constexpr int AR = MF * MF / 64;               // accumulator values per lane and block
    static constexpr int KW = 512 / MF;                   // k per MFMA (16 or 32)
    static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BK * BN * 2;
    static constexpr int A_PER_THREAD = BM * (BK / 8) / NT;   // 16-byte slots
    static constexpr int B_PER_THREAD = BK * (BN / 8) / NT;
    static constexpr int BCH = BN / 8;                    // 16-byte chunks per B row
    static constexpr int PER_STAGE = A_PER_THREAD + B_PER_THREAD;   // loads per thread
};

// ST stages of A and B tiles in LDS: two (double buffering, one tile in
// flight during the MFMAs) or a ring of three or four (ST - 1 tiles in
// flight) for grids of at most one workgroup per CU, where no other
// workgroup's MFMAs cover the wait for a tile.
template <int BM, int BN, int ST, int KS, int MF, bool CBF16>
__global__ __launch_bounds__(NT, 2) void gemm_kernel(GArgs args)
{
    using C = Cfg<BM, BN, KS, MF>;
    using Acc = typename std::conditional<MF == 32, f32x16, f32x4>::type;
    static_assert(KS == 1 || ((KS == 2 || KS == 4) && C::A_BYTES == 16384 &&
                              C::B_BYTES == 16384 &&
                              C::FM * C::FN * C::AR * 256 * C::WPG == 65536),
                  "a group's sums fill the four 16 KB stage buffers");
    static_assert(ST == 2 || (ST <= 4 && 2 * C::PER_STAGE < 16), "stage count / vmcnt range");
    static_assert((BK / C::KW) % KS == 0, "each group takes whole k-steps of every K step");
    __shared__ __attribute__((aligned(16))) unsigned char abuf[ST][C::A_BYTES];
    __shared__ __attribute__((aligned(16))) unsigned char bbuf[ST][C::B_BYTES];
    unsigned char *const a0 = abuf[0], *const a1 = abuf[1];
    unsigned char *const b0 = bbuf[0], *const b1 = bbuf[1];

    const GArgs &a = args;
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int col = lane % MF, half = lane / MF;   // lane's column of a block; its k part

    // XCD-contiguous logical tile index, row-major over the tiles of C
    const int per = a.n_wg / NXCD, rem = a.n_wg % NXCD;
    const int xcd = blockIdx.x % NXCD, idx = blockIdx.x / NXCD;
    const int t = xcd * per + (xcd < rem ? xcd : rem) + idx;
    // grouped order: GROUP_M consecutive logical tiles walk down a column of
    // tiles before moving right, so the workgroups resident on an XCD cover
    // a GROUP_M x (resident / GROUP_M) block of C and share its A and B
    // panels in that XCD's L2
    int tm = t / a.tiles_n, tn = t % a.tiles_n;
    if ((a.M / BM) % GROUP_M == 0) {
        const int per_group = GROUP_M * a.tiles_n;
        const int grp = t / per_group, w = t % per_group;
        tm = grp * GROUP_M + w % GROUP_M;
        tn = w / GROUP_M;
    }
    const int m0 = tm * BM, n0 = tn * BN;
    const int cw = KS == 1 ? wave & 3 : wave % C::WPG;    // column of the wave's block
    const int wm = KS == 1 ? (wave >> 2) * C::WM : 0, wn = cw * C::WN;
    const int kg = KS == 1 ? 0 : wave_u / C::WPG;          // this wave's share of each K step

    // per-lane DMA source offsets within a stage's tiles.  A slot
    // i*NT + 64w + l is row s / 8, stored chunk s % 8 (fetched from chunk
    // (s % 8) ^ a_swz(row)); B slot s is row s / BCH, stored chunk s % BCH
    // (fetched from chunk (s % BCH) ^ b_swz(row)).
    uint32_t a_off[C::A_PER_THREAD], b_off[C::B_PER_THREAD];
#pragma unroll
    for (int i = 0; i < C::A_PER_THREAD; ++i) {
        const int s = i * NT + wave_u * 64 + lane;
        const int r = s / 8, sc = s % 8;
        a_off[i] = (uint32_t)r * a.K * 2 + 16 * (sc ^ a_swz(r));
    }
#pragma unroll
    for (int i = 0; i < C::B_PER_THREAD; ++i) {
        const int s = i * NT + wave_u * 64 + lane;
        const int r = s / C::BCH, sc = s % C::BCH;
        b_off[i] = (uint32_t)r * a.N * 2 + 16 * (sc ^ b_swz<MF>(r));
    }

    auto dma = [&](int kt, unsigned char *as, unsigned char *bs) {
        const int k0 = kt * BK;
        const u32x4s ra = buffer_rsrc(a.A + (size_t)m0 * a.K + k0,
                                      (uint32_t)((BM - 1) * a.K + BK) * 2);
        const u32x4s rb = buffer_rsrc(a.B + (size_t)k0 * a.N + n0,
                                      (uint32_t)((BK - 1) * a.N + BN) * 2);
        const uint32_t la = lds_addr(as), lb = lds_addr(bs);
#pragma unroll
        for (int i = 0; i < C::A_PER_THREAD; ++i)
            dma16(la + (i * NT + wave_u * 64) * 16, a_off[i], ra);
#pragma unroll
        for (int i = 0; i < C::B_PER_THREAD; ++i)
            dma16(lb + (i * NT + wave_u * 64) * 16, b_off[i], rb);
    };

    Acc acc[C::FM][C::FN];
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j)
#pragma unroll
            for (int r = 0; r < C::AR; ++r)
                acc[i][j][r] = 0.f;

    // B operand transpose-read addressing (per 16-lane group g = lane / 16,
    // s = lane % 16).  MF = 32: rows 16ks + 8(g >> 1) + (s >> 2) and + 4,
    // columns 16(g & 1) + 4(s & 3) of each 32-column block: the lane then
    // holds 8 consecutive k of one column, k-slot t <-> k = 16ks + 8 half + t.
    // MF = 16: rows 32ks + 8g + (s >> 2) and + 4, columns 4(s & 3) of each
    // 16-column block: k-slot t <-> k = 32ks + 8g + t.
    const int g = lane >> 4, sl = lane & 15;
    const int b_row = MF == 32 ? 8 * (g >> 1) + (sl >> 2) : 8 * g + (sl >> 2);
    const int b_col = MF == 32 ? 16 * (g & 1) + 4 * (sl & 3) : 4 * (sl & 3);

    auto compute = [&](const unsigned char *as, const unsigned char *bs) {
#pragma unroll
        for (int kq = 0; kq < BK / C::KW / KS; ++kq) {
            const int ks = kg * (BK / C::KW / KS) + kq;
            bf16x8 av[C::FM], bv[C::FN];
#pragma unroll
            for (int i = 0; i < C::FM; ++i) {
                // lane: row col of the block, k (KW ks + 8 half ..) = chunk
                // (KW / 8) ks + half of the row
                const int r = wm + MF * i + col;
                av[i] = *(const bf16x8 *)(as + r * (BK * 2) +
                                          16 * (((C::KW / 8) * ks + half) ^ a_swz(r)));
            }
#pragma unroll
            for (int j = 0; j < C::FN; ++j) {
                const int n = wn + MF * j + b_col;
                const int r0 = C::KW * ks + b_row, r1 = r0 + 4;
                const unsigned char *p0 =
                    bs + r0 * (BN * 2) + 16 * ((n >> 3) ^ b_swz<MF>(r0)) + 2 * (n & 7);
                const unsigned char *p1 =
                    bs + r1 * (BN * 2) + 16 * ((n >> 3) ^ b_swz<MF>(r1)) + 2 * (n & 7);
                const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p0);
                const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p1);
                const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
                bv[j] = __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
            }
#pragma unroll
            for (int i = 0; i < C::FM; ++i)
#pragma unroll
                for (int j = 0; j < C::FN; ++j)
                    acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
        }
    };

    const int n_kt = a.K / BK;
    if constexpr (ST == 2) {
        dma(0, a0, b0);
        wait_dma_all();
        __syncthreads();
        int kt = 0;
        for (; kt + 1 < n_kt; kt += 2) {
            dma(kt + 1, a1, b1);
            compute(a0, b0);
            wait_dma_all();
            __syncthreads();
            if (kt + 2 < n_kt)
                dma(kt + 2, a0, b0);
            compute(a1, b1);
            wait_dma_all();
            __syncthreads();
        }
        if (kt < n_kt)
            compute(a0, b0);
    } else {
        // ring: K step kt lives in stage kt % ST.  Before step kt, wait for
        // its loads (those of the up to ST - 2 later steps already issued
        // may stay in flight), then one barrier: every thread's part of
        // step kt is in LDS and every wave is done with step kt - 1, whose
        // stage takes step kt + ST - 1.
#pragma unroll
        for (int st = 0; st < ST - 1; ++st)
            if (st < n_kt)
                dma(st, abuf[st], bbuf[st]);
        for (int kt = 0; kt < n_kt; ++kt) {
            const int ahead = min(ST - 2, n_kt - 1 - kt);
            if (ahead >= 2)
                wait_dma_upto<2 * C::PER_STAGE>();
            else if (ahead == 1)
                wait_dma_upto<C::PER_STAGE>();
            else
                wait_dma_all();
            __syncthreads();
            const int nx = kt + ST - 1;
            if (nx < n_kt)
                dma(nx, abuf[nx % ST], bbuf[nx % ST]);
            compute(abuf[kt % ST], bbuf[kt % ST]);
        }
    }

    if constexpr (KS > 1) {
        // group 0 adds the other groups' sums, one group per round, in
        // group order.  Accumulator block k = i FN + j of the wave in
        // column cw goes, lane-major, to piece k (AR KB) of the wave's
        // FM FN AR KB of the four 16 KB stage buffers, in buffer order.
        constexpr int PB = C::AR * 256;                         // bytes per block
        constexpr int NB = C::FM * C::FN * PB / 16384;          // 16 KB buffers per wave
        auto piece = [&](int k) {
            const int bi = cw * NB + (k * PB) / 16384;
            unsigned char *base = bi == 0 ? abuf[0] : bi == 1 ? abuf[1] : bi == 2 ? bbuf[0] : bbuf[1];
            return (float *)(base + (k * PB) % 16384);
        };
        __syncthreads();   // every wave is done with the stage buffers
#pragma unroll
        for (int g = 1; g < KS; ++g) {
            if (kg == g) {
#pragma unroll
                for (int i = 0; i < C::FM; ++i)
#pragma unroll
                    for (int j = 0; j < C::FN; ++j) {
                        float *p = piece(i * C::FN + j);
#pragma unroll
                        for (int r = 0; r < C::AR; ++r)
                            p[r * 64 + lane] = acc[i][j][r];
                    }
            }
            __syncthreads();
            if (kg == 0) {
#pragma unroll
                for (int i = 0; i < C::FM; ++i)
#pragma unroll
                    for (int j = 0; j < C::FN; ++j) {
                        const float *p = piece(i * C::FN + j);
#pragma unroll
                        for (int r = 0; r < C::AR; ++r)
                            acc[i][j][r] += p[r * 64 + lane];
                    }
            }
            if (g + 1 < KS)
                __syncthreads();   // read before the next group writes
        }
        if (kg != 0)
            return;
    }

    // epilogue: lane holds column wn + MF j + col, rows wm + MF i +
    // 8(r/4) + 4half + r%4 (MF = 32) or 4half + r (MF = 16) of the tile
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
            const int n = n0 + wn + MF * j + col;
#pragma unroll
            for (int r = 0; r < C::AR; ++r) {
                const int m = m0 + wm + MF * i + (MF == 32 ? 8 * (r >> 2) : 0) + 4 * half + (r & 3);
                if (CBF16)
                    ((uint16_t *)a.C)[(size_t)m * a.N + n] =
                        (uint16_t)pack_bf16(acc[i][j][r], 0.f);
                else
                    ((float *)a.C)[(size_t)m * a.N + n] = acc[i][j][r];
            }
        }
}

// ---- M = 1: the matrix-vector product C[n] = sum_k a[k] B[k][n] ----------
// (the paper's V0-V7 shapes).  B is read once and every byte of it feeds one
// multiply-add, so this is HBM-bound and runs on the vector ALUs.  A
// workgroup of 16 waves owns a strip of COLS columns (COLS * 2 contiguous
// bytes of each B row); a lane reads 16 bytes (8 columns) of a row, so one
// load instruction covers RPL = 512 / COLS full row segments.  Rows are taken
// in groups of 8 (SPLIT: the groups of key range blockIdx.y of gridDim.y),
// split evenly over the waves; a wave walks its groups RPL
// (or 2 RPL) at a time, lane g (of RPL) taking all 8 rows of group gi + g
// (or 16 rows of groups gi + 2g, gi + 2g + 1), so that its values of a are
// 16-byte loads.  Partial sums meet in LDS and COLS
// threads add them in a fixed order (results do not depend on timing); with
// SPLIT the strip's sum over its range goes, in fp32, to row blockIdx.y of
// the workspace C [gridDim.y][N] for gemv_combine_kernel.
constexpr int GV_WAVES = 16;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
// B is read exactly once per call.  When it is larger than the 256 MB
// Infinity Cache it goes through non-temporal loads (measured 5.1 -> 5.7
// TB/s at V0, 6.1 -> 6.8 at V3, 4.0 -> 4.2 at V7 against ordinary loads);
// a smaller B is read with ordinary loads, so that calls repeated on the
// same matrix can find it there (V5, 170 MB: 6.1 TB/s, 4.1 non-temporal).
template <bool NT>
__device__ __forceinline__ u32x4 ld_b(const uint16_t *p)
{
    if (NT)
        return __builtin_nontemporal_load((const u32x4 *)p);
    return *(const u32x4 *)p;
}
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

template <int COLS, bool NT, bool CBF16, bool SPLIT>
__global__ __launch_bounds__(64 * GV_WAVES) void gemv_kernel(const uint16_t *A, const uint16_t *B,
                                                              void *C, int N, int K)
{
    constexpr int LPR = COLS / 8;       // lanes per row segment
    constexpr int RPL = 64 / LPR;       // row segments per load instruction
    static_assert(RPL >= 1 && 8 % RPL == 0, "strip width");
    __shared__ float red[GV_WAVES][RPL][COLS];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n0 = blockIdx.x * COLS;
    const int g = lane / LPR;
    const int c8 = (lane % LPR) * 8;    // this lane's first column in the strip
    int gb = 0, groups = K / 8;
    if (SPLIT) {
        const int all = groups, sp = blockIdx.y, ns = gridDim.y;
        gb = (int)((int64_t)all * sp / ns);
        groups = (int)((int64_t)all * (sp + 1) / ns) - gb;
    }
    const int g0 = gb + (int)((int64_t)groups * wave / GV_WAVES);
    const int g1 = gb + (int)((int64_t)groups * (wave + 1) / GV_WAVES);

    float acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
        acc[i] = 0.f;
    auto fma8 = [&](float x, const u32x4 &bv) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            acc[2 * i] = __builtin_fmaf(x, bf16_lo(bv[i]), acc[2 * i]);
            acc[2 * i + 1] = __builtin_fmaf(x, bf16_hi(bv[i]), acc[2 * i + 1]);
        }
    };
    int gi = g0;
    // 64-column strips: two groups (16 rows) per lane and step, 16 loads in
    // flight per lane; 256-column strips: one group
    constexpr int GPL = COLS == 64 ? 2 : 1;
    for (; gi + GPL * RPL <= g1; gi += GPL * RPL) {
        const size_t r0 = (size_t)8 * (gi + GPL * g);
        const uint16_t *bp = B + r0 * N + n0 + c8;
        u32x4 bv[8 * GPL];
#pragma unroll
        for (int u = 0; u < 8 * GPL; ++u)
            bv[u] = ld_b<NT>(bp + (size_t)u * N);
        u32x4 av[GPL];
#pragma unroll
        for (int q = 0; q < GPL; ++q)
            av[q] = *(const u32x4 *)(A + r0 + 8 * q);
#pragma unroll
        for (int u = 0; u < 8 * GPL; ++u) {
            const uint32_t w = av[u >> 3][(u & 7) >> 1];
            fma8((u & 1) ? bf16_hi(w) : bf16_lo(w), bv[u]);
        }
    }
    // then single groups per lane while RPL of them are left
    for (; gi + RPL <= g1; gi += RPL) {
        const size_t r0 = (size_t)8 * (gi + g);
        const uint16_t *bp = B + r0 * N + n0 + c8;
        u32x4 bv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            bv[u] = ld_b<NT>(bp + (size_t)u * N);
        const u32x4 av = *(const u32x4 *)(A + r0);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            fma8((u & 1) ? bf16_hi(av[u >> 1]) : bf16_lo(av[u >> 1]), bv[u]);
    }
    // fewer than RPL groups left: one group at a time, lane g on its rows
    // g, g + RPL, ... of the group
    for (; gi < g1; ++gi)
#pragma unroll
        for (int h = 0; h < 8 / RPL; ++h) {
            const size_t r = (size_t)8 * gi + h * RPL + g;
            fma8(__uint_as_float((uint32_t)A[r] << 16), ld_b<NT>(B + r * N + n0 + c8));
        }

#pragma unroll
    for (int i = 0; i < 8; ++i)
        red[wave][g][c8 + i] = acc[i];
    __syncthreads();
    if (tid < COLS) {
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < GV_WAVES; ++w)
#pragma unroll
            for (int r = 0; r < RPL; ++r)
                sum += red[w][r][tid];
        if (SPLIT)
            ((float *)C)[(size_t)blockIdx.y * N + n0 + tid] = sum;
        else if (CBF16)
            ((uint16_t *)C)[n0 + tid] = (uint16_t)pack_bf16(sum, 0.f);
        else
            ((float *)C)[n0 + tid] = sum;
    }
}

// The merge of gemv_bf16_split: C[n] = W[0][n] + W[1][n] + ... + W[S-1][n],
// added in that order (fp32), then rounded once if C is bf16.
constexpr int GV_COMBINE = 256;
template <bool CBF16>
__global__ __launch_bounds__(GV_COMBINE) void gemv_combine_kernel(const float *W, void *C, int N,
                                                                  int S)
{
    const int n = blockIdx.x * GV_COMBINE + threadIdx.x;
    if (n >= N)
        return;
    const float *w = W + n;
    float sum = w[0];
    // up to eight rows' loads in flight before their adds (the split counts
    // in use are 2-9: one or two round trips instead of one per row)
    for (int s = 1; s < S; s += 8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            v[u] = s + u < S ? w[(size_t)(s + u) * N] : 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (s + u < S)
                sum += v[u];
    }
    if (CBF16)
        ((uint16_t *)C)[n] = (uint16_t)pack_bf16(sum, 0.f);
    else
        ((float *)C)[n] = sum;
}

// Strips of 256 columns (512-byte row segments) stream B faster than
// 128-byte ones, but only when there are enough of them to give most CUs a
// workgroup: measured 5.5-6.2 TB/s against 4.5-5.0 on the paper's N >= 36864
// shapes, and 2.6-3.2 TB/s against 4.1-5.8 on N <= 16384.
template <bool NT, bool CBF16>
hipError_t launch_gemv(const uint16_t *a, const uint16_t *b, void *C, int N, int K, hipStream_t s)
{
    if (N % 256 == 0 && N / 256 >= 144)
        hipLaunchKernelGGL((gemv_kernel<256, NT, CBF16, false>), dim3(N / 256), dim3(64 * GV_WAVES),
                           0, s, a, b, C, N, K);
    else
        hipLaunchKernelGGL((gemv_kernel<64, NT, CBF16, false>), dim3(N / 64), dim3(64 * GV_WAVES),
                           0, s, a, b, C, N, K);
    return hipGetLastError();
}

// K split into S ranges: 256-column strips wherever N allows (their rows
// stream faster), S workgroups per strip writing fp32 partial sums to W
// [S][N], then the merge.
template <bool NT>
hipError_t launch_gemv_split(const uint16_t *a, const uint16_t *b, void *C, bool c_bf16, int N,
                             int K, int S, float *W, hipStream_t s)
{
    if (N % 256 == 0)
        hipLaunchKernelGGL((gemv_kernel<256, NT, false, true>), dim3(N / 256, S),
                           dim3(64 * GV_WAVES), 0, s, a, b, (void *)W, N, K);
    else
        hipLaunchKernelGGL((gemv_kernel<64, NT, false, true>), dim3(N / 64, S), dim3(64 * GV_WAVES),
                           0, s, a, b, (void *)W, N, K);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const dim3 grid((N + GV_COMBINE - 1) / GV_COMBINE);
    if (c_bf16)
        hipLaunchKernelGGL(gemv_combine_kernel<true>, grid, dim3(GV_COMBINE), 0, s, W, C, N, S);
    else
        hipLaunchKernelGGL(gemv_combine_kernel<false>, grid, dim3(GV_COMBINE), 0, s, W, C, N, S);
    return hipGetLastError();
}

// B larger than the 256 MB Infinity Cache: non-temporal loads
bool gemv_nt(int N, int K) { return (size_t)K * N * 2 > ((size_t)256 << 20); }

hipError_t run_gemv(const void *A, const void *B, void *C, bool c_bf16, int N, int K, hipStream_t s)
{
    const auto a = (const uint16_t *)A, b = (const uint16_t *)B;
    if (gemv_nt(N, K))
        return c_bf16 ? launch_gemv<true, true>(a, b, C, N, K, s)
                      : launch_gemv<true, false>(a, b, C, N, K, s);
    return c_bf16 ? launch_gemv<false, true>(a, b, C, N, K, s)
                  : launch_gemv<false, false>(a, b, C, N, K, s);
}


constexpr int GV_MAX_SPLITS = 64;

bool misaligned(const void *p) { return ((uintptr_t)p & 15u) != 0; }

bool overlaps(const void *p, size_t pn, const void *q, size_t qn)
{
    const uintptr_t x = (uintptr_t)p, y = (uintptr_t)q;
    return x < y + qn && y < x + pn;
}

// 16 x 16 blocks (v_mfma_f32_16x16x32_bf16) wherever a group's share of a
// K step holds whole 32-wide k-steps: under the board's power limit that
// MFMA form holds a higher clock than 32 x 32 x 16 (M5 1314 -> 1346-1359,
// M1 1274-1297 -> 1333-1348, M4 1150 -> 1177 TFLOP/s); four groups share a
// K step of 64 as 16-wide k-steps, so their tiles keep 32 x 32 blocks.
template <int BM, int BN, int ST, int KS>
hipError_t launch(GArgs &a, bool c_bf16, hipStream_t s)
{
    constexpr int MF = (BK / 32) % KS == 0 ? 16 : 32;
    a.tiles_n = a.N / BN;
    a.n_wg = (a.M / BM) * a.tiles_n;
    if (c_bf16)
        hipLaunchKernelGGL((gemm_kernel<BM, BN, ST, KS, MF, true>), dim3(a.n_wg), dim3(NT), 0, s, a);
    else
        hipLaunchKernelGGL((gemm_kernel<BM, BN, ST, KS, MF, false>), dim3(a.n_wg), dim3(NT), 0, s, a);
    return hipGetLastError();
}

}  // namespace

extern "C" {

ta_status gemm_bf16(const void *A, const void *B, void *C, int c_bf16, int M, int N, int K,
                    void *stream)
{
    if (!A || !B || !C)
        return TA_ERR_NULL_POINTER;
    if (M < 1 || N < 1 || K < 1)
        return TA_ERR_INVALID_SHAPE;
    const bool gemv = M == 1;
    if (gemv ? (N % 64 || K % 8) : (M % 128 || N % 128 || K % BK))
        return TA_ERR_UNSUPPORTED;
    // the tiled kernel: 32-bit offsets within a workgroup's tiles and buffer
    // ranges (the matrix-vector kernel addresses with 64-bit pointers)
    if (!gemv && ((int64_t)K * N * 2 >= (1ll << 31) || (int64_t)M * K >= (1ll << 40) ||
                  (int64_t)256 * K * 2 >= (1ll << 31)))
        return TA_ERR_INVALID_SHAPE;
    if (misaligned(A) || misaligned(B) || misaligned(C))
        return TA_ERR_MISALIGNED;
    const size_t a_bytes = (size_t)M * K * 2, b_bytes = (size_t)K * N * 2;
    const size_t c_bytes = (size_t)M * N * (c_bf16 ? 2 : 4);
    if (overlaps(C, c_bytes, A, a_bytes) || overlaps(C, c_bytes, B, b_bytes))
        return TA_ERR_ALIASING;
    GArgs a;
    a.A = (const uint16_t *)A;
    a.B = (const uint16_t *)B;
    a.C = C;
    a.M = M;
    a.N = N;
    a.K = K;
    hipStream_t s = (hipStream_t)stream;
    if (gemv) {
        const hipError_t e = run_gemv(A, B, C, c_bf16 != 0, N, K, s);
        return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH;
    }
    // 256 x 256 tiles when they give at least one workgroup per CU
    // (128 x 128 tiles: with at most one workgroup per CU, a ring of four
    // stages and K steps split over four groups of two waves (169 registers:
    // two waves per SIMD); otherwise two stages and two groups of four (at
    // most 128 registers, so that two workgroups share a CU))
    const bool big = M % 256 == 0 && N % 256 == 0 && (int64_t)(M / 256) * (N / 256) >= 256;
    const bool ring = (int64_t)(M / 128) * (N / 128) <= 256;
    const hipError_t e = big    ? launch<256, 256, 2, 1>(a, c_bf16 != 0, s)
                         : ring ? launch<128, 128, 4, 4>(a, c_bf16 != 0, s)
                                : launch<128, 128, 2, 2>(a, c_bf16 != 0, s);
    return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH;
}

ta_status gemv_bf16_split(const void *A, const void *B, void *C, int c_bf16, int N, int K,
                          int num_splits, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!A || !B || !C)
        return TA_ERR_NULL_POINTER;
    if (N < 1 || K < 1 || num_splits < 1 || num_splits > GV_MAX_SPLITS)
        return TA_ERR_INVALID_SHAPE;
    if (N % 64 || K % 8)
        return TA_ERR_UNSUPPORTED;
    if (misaligned(A) || misaligned(B) || misaligned(C))
        return TA_ERR_MISALIGNED;
    const size_t a_bytes = (size_t)K * 2, b_bytes = (size_t)K * N * 2;
    const size_t c_bytes = (size_t)N * (c_bf16 ? 2 : 4);
    if (overlaps(C, c_bytes, A, a_bytes) || overlaps(C, c_bytes, B, b_bytes))
        return TA_ERR_ALIASING;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (num_splits == 1) {
        e = run_gemv(A, B, C, c_bf16 != 0, N, K, s);
    } else {
        const size_t w_bytes = (size_t)num_splits * N * 4;
        if (!workspace || workspace_bytes < w_bytes)
            return TA_ERR_WORKSPACE;
        if (misaligned(workspace))
            return TA_ERR_MISALIGNED;
        if (overlaps(workspace, w_bytes, A, a_bytes) || overlaps(workspace, w_bytes, B, b_bytes) ||
            overlaps(workspace, w_bytes, C, c_bytes))
            return TA_ERR_ALIASING;
        const auto a = (const uint16_t *)A, b = (const uint16_t *)B;
        const auto w = (float *)workspace;
        e = gemv_nt(N, K) ? launch_gemv_split<true>(a, b, C, c_bf16 != 0, N, K, num_splits, w, s)
                          : launch_gemv_split<false>(a, b, C, c_bf16 != 0, N, K, num_splits, w, s);
    }
    return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH;
}

ta_status gemv_split_workspace_bytes(int N, int num_splits, size_t *bytes)
{
    if (!bytes)
        return TA_ERR_NULL_POINTER;
    if (N < 1 || num_splits < 1 || num_splits > GV_MAX_SPLITS)
        return TA_ERR_INVALID_SHAPE;
    *bytes = num_splits > 1 ? (size_t)num_splits * N * 4 : 0;
    return TA_OK;
}

// The split count whose workgroups fill their last round of CU slots most
// evenly (one slot per CU per round; two 16-wave workgroups fit a CU), up
// to two rounds, keeping at least 1024 rows per split; on a tie the fewer
// workgroups.  Strips are 256 columns where N % 256 == 0, else 64; one
// split runs the unsplit kernel, whose strips are 64 columns unless there
// are 144 or more of 256, so with 256-column splits available it only
// counts when that holds.  (Measured, the paper's V0-V7 shapes: a count
// just past a multiple of 256 is 10-26 % slower than one just below it.)
ta_status gemv_split_heuristic(int N, int K, int *num_splits)
{
    if (!num_splits)
        return TA_ERR_NULL_POINTER;
    if (N < 1 || K < 1)
        return TA_ERR_INVALID_SHAPE;
    constexpr int64_t CUS = 256;
    const bool wide = N % 256 == 0;
    const int64_t strips = wide ? N / 256 : ((int64_t)N + 63) / 64;
    // is w1 workgroups' last round fuller than w2's
    auto fuller = [](int64_t w1, int64_t w2) {
        const int64_t r1 = CUS * ((w1 + CUS - 1) / CUS), r2 = CUS * ((w2 + CUS - 1) / CUS);
        return w1 * r2 > w2 * r1;
    };
    int n = 1;
    int64_t best = !wide || strips >= 144 ? strips : -1;
    for (int sp = 2; sp <= GV_MAX_SPLITS && strips * sp <= 2 * CUS && K / sp >= 1024; ++sp)
        if (best < 0 || fuller(strips * sp, best)) {
            n = sp;
            best = strips * sp;
        }
    *num_splits = n;
    return TA_OK;
}

}  // extern "C"
