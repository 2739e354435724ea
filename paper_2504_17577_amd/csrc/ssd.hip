// Mamba-2 state-space-duality (SSD) chunk kernels for gfx950 (MI355X): the
// chunk-state and chunk-scan functions the paper benchmarks as its linear
// attention workload (Section "Numerical Experiments", paragraph "Linear
// Attention Performance"; shapes in the appendix table "Linear Attention
// shapes in our benchmark"), plus the state passing and per-chunk C B^T
// steps that complete the chained forward pass.
//
// For batch b, head h (group g = h / (H/G)) and chunk c of Q = 256 positions,
// with the cumulative log-decay a_l = sum_{l' <= l} dt_{l'} A_h inside the
// chunk:
//   chunk state    S_c[p][n]  = sum_l exp(a_last - a_l) dt_l x_l[p] Bm_l[n]
//   state passing  H_c = exp(a_last(c)) H_{c-1} + S_c, H_{-1} = 0; chunk c
//                  enters with H_{c-1}
//   chunk matrix   cb[l][s]   = Cm_l . Bm_s
//   chunk scan     y_l[p] = exp(a_l) sum_n H_{c-1}[p][n] Cm_l[n]
//                         + sum_{s <= l} cb[l][s] exp(a_l - a_s) dt_s x_s[p]
//                         + D_h x_l[p]
// The design is this library's own for CDNA4:
//  * One workgroup of four wave64s per (batch, chunk, head).  The workgroup
//    forms the chunk's cumulative decay itself (a 256-wide prefix sum of
//    dt * A), so the functions take the raw dt and A.
//  * Every contraction runs on v_mfma_f32_32x32x16_bf16 with fp32
//    accumulation.  The decay- and dt-weighted operand (x for the chunk
//    state, the masked cb matrix for the chunk scan) and the fp32 entering
//    state are rounded to bf16 (nearest even) once, right before the MFMA.
//  * Outputs are computed transposed (S^T, y^T), so that each lane of the
//    32x32 accumulator layout owns four consecutive elements of a row of the
//    row-major result and stores them as one 16-byte write.
//  * Operands that must be read along the sequence (columns of x and Bm)
//    come from LDS through the gfx950 transpose read ds_read_b64_tr_b16;
//    rows are read with ds_read_b128 or straight from global memory.
//  * Workgroup ids are remapped so that each XCD runs whole (batch, chunk)
//    groups of heads: the chunk's Bm, Cm and cb, shared by all its heads,
//    stay in that XCD's L2.
#include <hip/hip_runtime.h>
#include <math.h>
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

constexpr int SQ = 256;       // chunk length
constexpr int SP = 64;        // head dim
constexpr int SN = 128;       // state dim
constexpr int NT = 256;       // threads per workgroup
constexpr int NXCD = 8;
constexpr float LOG2E = 1.44269504088896340736f;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// hardware workgroup id -> logical id: XCD x (which receives ids x, x + 8,
// ...) gets the contiguous logical range [x * per, ...)
__device__ __forceinline__ int xcd_logical(int bid, int n_wg)
{
    const int per = n_wg / NXCD, rem = n_wg % NXCD;
    const int xcd = bid % NXCD, idx = bid / NXCD;
    return xcd * per + (xcd < rem ? xcd : rem) + idx;
}

// inclusive prefix sum over the workgroup's 256 threads (ascending tid)
__device__ float block_scan(float v, float *wsum)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const float u = __shfl_up(v, d, 64);
        if (lane >= d)
            v += u;
    }
    if (lane == 63)
        wsum[wave] = v;
    __syncthreads();
    float off = 0.f;
    for (int w = 0; w < wave; ++w)
        off += wsum[w];
    return v + off;
}

// 16-byte chunk c of row r of a tile with 256-byte rows (128 bf16), stored
// at c ^ swz: conflict-free for the transpose reads (4 rows x 64 bytes per
// half wave) and for 32-row ds_read_b128 operand reads
__device__ __forceinline__ int swz_tr256(int r) { return 4 * (r & 3); }
__device__ __forceinline__ int swz_row256(int r) { return r & 15; }
// 128-byte rows (64 bf16)
__device__ __forceinline__ int swz_tr128(int r) { return 4 * ((r >> 1) & 1); }

// Transpose read of an MFMA operand from a row-major bf16 tile: lane l gets
// the 8 k-slots {k0 + 4h + t, k0 + 8 + 4h + t : t < 4} (h = l / 32) of
// column col0 + l % 32.  Two ds_read_b64_tr_b16: each group of 16 lanes reads
// a 4 x 16 block (rows k0 + 4h (+8) + s/4, columns col0 + 16((l>>4)&1) +
// 4(s&3) for s = l % 16) and the transpose hands lane s column s of it.
template <int ROWB, int (*SWZ)(int)>
__device__ __forceinline__ bf16x8 tr_operand(const unsigned char *tile, int k0, int col0, int lane)
{
    const int gq = lane >> 4, sl = lane & 15, h = lane >> 5;
    const int r0 = k0 + 4 * h + (sl >> 2), r1 = r0 + 8;
    const int col = col0 + 16 * (gq & 1) + 4 * (sl & 3);
    const int bin = (2 * col) & 15;
    const unsigned char *p0 = tile + r0 * ROWB + (((col >> 3) ^ SWZ(r0)) * 16) + bin;
    const unsigned char *p1 = tile + r1 * ROWB + (((col >> 3) ^ SWZ(r1)) * 16) + bin;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p0);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p1);
    const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
    return __builtin_bit_cast(bf16x8, u32x4{l2[0], l2[1], h2[0], h2[1]});
}

// Loads of sequence positions past L read the last real position instead
// (always a valid address) and are zeroed after the load: no branch, so the
// compiler can issue a whole batch of them before the first wait.
__device__ __forceinline__ u32x4 load_row16(const uint16_t *p, bool keep)
{
    const u32x4 v = *(const u32x4 *)p;
    return keep ? v : u32x4{0u, 0u, 0u, 0u};
}

// The streams that are read or written exactly once per call (x, the
// entering states, the outputs) go through non-temporal accesses when they
// add up to more than twice the 256 MB Infinity Cache (STREAM); the operands
// that every head of a group re-reads (Bm, Cm, cb) stay ordinary.  Measured
// at B=64 L=2048: chunk scan 4.14 -> 4.37 TB/s, chunk state 4.40 -> 4.74.
// Smaller calls keep ordinary accesses, so that calls repeated on the same
// tensors can find part of them there (B=1 L=8192, 134 and 268 MB: chunk
// state 4.46 TB/s, 3.65 non-temporal; chunk scan 3.40, 3.21).
template <bool STREAM>
__device__ __forceinline__ u32x4 ld_once(const uint16_t *p)
{
    if (STREAM)
        return __builtin_nontemporal_load((const u32x4 *)p);
    return *(const u32x4 *)p;
}
template <bool STREAM>
__device__ __forceinline__ f32x4 ld_once(const float *p)
{
    if (STREAM)
        return __builtin_nontemporal_load((const f32x4 *)p);
    return *(const f32x4 *)p;
}
template <bool STREAM>
__device__ __forceinline__ void st_once(float *p, f32x4 v)
{
    if (STREAM)
        __builtin_nontemporal_store(v, (f32x4 *)p);
    else
        *(f32x4 *)p = v;
}
constexpr size_t STREAM_BYTES = (size_t)512 << 20;

struct SsdShape {
    int B, L, H, G, nc;
    int hpg;   // H / G
};

// ---------------------------------------------------------------------------
// chunk state: S^T[n][p] = sum_l Bm_l[n] (x_l[p] w_l),  w_l = exp(a_last - a_l) dt_l

struct StateArgs {
    SsdShape s;
    const uint16_t *x, *Bm;
    const float *dt, *A;
    float *states;
};

// One workgroup per (batch, chunk, HPW heads of one group).  The heads share
// the Bm operand (read once for all of them), and a position's x slice of
// the HPW heads is HPW * 128 contiguous bytes, read whole: two heads per
// workgroup measured 4.73 -> 5.35 TB/s at B=64 L=2048 against one (128-byte
// row pieces, Bm read per head), four heads 5.25 (two waves per SIMD).
// Positions are staged in passes of 32 (Bm 8 KB + HPW weighted x tiles of 4
// KB in LDS, so several workgroups share a CU and cover each other's memory
// latency); the global loads of pass k + 1 are issued into registers before
// the MFMAs of pass k.  The result rows go through LDS, 32 rows of S (512
// bytes each) at a time, so that a store instruction covers two whole rows;
// 16-byte chunk q of staged row r sits at chunk q ^ r.
template <int HPW, bool STREAM>
__global__ __launch_bounds__(NT, HPW >= 4 ? 2 : HPW == 2 ? 4 : 6) void chunk_state_kernel(StateArgs args)
{
    const StateArgs &a = args;
    constexpr int PASS = 32;
    constexpr int NPASS = SQ / PASS;
    constexpr int XT = PASS * SP * 2;                       // one head's x tile of a pass
    constexpr int PASS_BYTES = PASS * SN * 2 + HPW * XT;
    constexpr int STG_BYTES = 32 * SN * 4;
    __shared__ __attribute__((aligned(16))) unsigned char smem[PASS_BYTES > STG_BYTES ? PASS_BYTES : STG_BYTES];
    unsigned char *const bt = smem;
    unsigned char *const xt = smem + PASS * SN * 2;
    __shared__ float wts[HPW][SQ];
    __shared__ float wsum[4];
    __shared__ float alast[HPW];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hgs = a.s.H / HPW;
    const int n_wg = a.s.B * a.s.nc * hgs;
    const int logical = xcd_logical(blockIdx.x, n_wg);
    const int h0 = (logical % hgs) * HPW;
    const int c = (logical / hgs) % a.s.nc;
    const int b = logical / (hgs * a.s.nc);
    const int g = h0 / a.s.hpg;

    const size_t brow = (size_t)a.s.G * SN;
    const size_t xrow = (size_t)a.s.H * SP;
    const int rb0 = tid >> 4, rb1 = (NT + tid) >> 4, cb_ = tid & 15;
    const uint16_t *bsrc = a.Bm + (size_t)b * a.s.L * brow + (size_t)g * SN + cb_ * 8;
    const uint16_t *xbase = a.x + (size_t)b * a.s.L * xrow + (size_t)h0 * SP;
    // x chunk i of this thread: row (i NT + tid) / (8 HPW), chunk (i NT + tid) % (8 HPW)
    u32x4 nb0, nb1, nx[HPW];
    auto load_pass = [&](int k) {
        const int p0 = c * SQ + k * PASS;
        nb0 = *(const u32x4 *)(bsrc + (size_t)min(p0 + rb0, a.s.L - 1) * brow);
        nb1 = *(const u32x4 *)(bsrc + (size_t)min(p0 + rb1, a.s.L - 1) * brow);
#pragma unroll
        for (int i = 0; i < HPW; ++i) {
            const int q = i * NT + tid, r = q / (8 * HPW), cc = q % (8 * HPW);
            nx[i] = ld_once<STREAM>(xbase + (size_t)min(p0 + r, a.s.L - 1) * xrow + cc * 8);
        }
    };
    load_pass(0);

    const int t = c * SQ + tid;
    const bool tv = t < a.s.L;
#pragma unroll
    for (int hi = 0; hi < HPW; ++hi) {
        const float dtv = a.dt[((size_t)b * a.s.L + min(t, a.s.L - 1)) * a.s.H + h0 + hi];
        const float dtl = tv ? dtv : 0.f;
        const float cum = block_scan(dtl * a.A[h0 + hi], wsum);
        if (tid == NT - 1)
            alast[hi] = cum;
        __syncthreads();   // alast visible; wsum free for the next head
        wts[hi][tid] = exp2f((alast[hi] - cum) * LOG2E) * dtl;
    }

    f32x16 acc[HPW][2];
#pragma unroll
    for (int hi = 0; hi < HPW; ++hi)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[hi][pb][r] = 0.f;

    for (int k = 0; k < NPASS; ++k) {
        __syncthreads();
        const int p0 = c * SQ + k * PASS;
        *(u32x4 *)(bt + rb0 * (SN * 2) + ((cb_ ^ swz_tr256(rb0)) * 16)) =
            p0 + rb0 < a.s.L ? nb0 : u32x4{0u, 0u, 0u, 0u};
        *(u32x4 *)(bt + rb1 * (SN * 2) + ((cb_ ^ swz_tr256(rb1)) * 16)) =
            p0 + rb1 < a.s.L ? nb1 : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < HPW; ++i) {
            const int q = i * NT + tid, r = q / (8 * HPW), cc = q % (8 * HPW);
            const int hi = cc / 8, pc = cc % 8;
            const float w = wts[hi][k * PASS + r];
            u32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] = pack_bf16(bf16_lo(nx[i][e]) * w, bf16_hi(nx[i][e]) * w);
            *(u32x4 *)(xt + hi * XT + r * (SP * 2) + ((pc ^ swz_tr128(r)) * 16)) = v;
        }
        __syncthreads();
        if (k + 1 < NPASS)
            load_pass(k + 1);
#pragma unroll
        for (int ks = 0; ks < PASS / 16; ++ks) {
            const bf16x8 av = tr_operand<SN * 2, swz_tr256>(bt, 16 * ks, 32 * wave, lane);
#pragma unroll
            for (int hi = 0; hi < HPW; ++hi)
#pragma unroll
                for (int pb = 0; pb < 2; ++pb) {
                    const bf16x8 bv = tr_operand<SP * 2, swz_tr128>(xt + hi * XT, 16 * ks, 32 * pb, lane);
                    acc[hi][pb] = mfma32(av, bv, acc[hi][pb]);
                }
        }
    }

    const int col = lane & 31, hl = lane >> 5;
#pragma unroll
    for (int hi = 0; hi < HPW; ++hi) {
        float *out = a.states + (((size_t)b * a.s.nc + c) * a.s.H + h0 + hi) * (SP * SN);
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
            __syncthreads();
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int q = 8 * wave + 2 * j + hl;
                *(float4 *)(smem + col * (SN * 4) + ((q ^ col) * 16)) =
                    float4{acc[hi][pb][4 * j], acc[hi][pb][4 * j + 1], acc[hi][pb][4 * j + 2],
                           acc[hi][pb][4 * j + 3]};
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = 8 * wave + 2 * i + hl;
                st_once<STREAM>(out + (32 * pb + r) * SN + 4 * col,
                                *(const f32x4 *)(smem + r * (SN * 4) + ((col ^ r) * 16)));
            }
        }
    }
}

// ---------------------------------------------------------------------------
// chunk scan: y^T[p][l] = exp(a_l) sum_n Hin[p][n] Cm_l[n]
//                         + sum_{s <= l} x_s[p] (cb[l][s] exp(a_l - a_s) dt_s)  + D x_l[p]

struct ScanArgs {
    SsdShape s;
    const uint16_t *x, *Cm;
    const float *cb, *dt, *A, *prev, *D;
    float *out;
};

template <bool STREAM>
__global__ __launch_bounds__(NT, 3) void chunk_scan_kernel(ScanArgs args)
{
    const ScanArgs &a = args;
    __shared__ __attribute__((aligned(16))) unsigned char xt[SQ * SP * 2];    // x rows, 32 KB
    __shared__ __attribute__((aligned(16))) unsigned char ht[SP * SN * 2];    // Hin (bf16), 16 KB
    __shared__ __attribute__((aligned(16))) float a2s[SQ];                    // log2-domain a_l
    __shared__ __attribute__((aligned(16))) float fs[SQ];                     // see below
    __shared__ float wsum[4];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n_wg = a.s.B * a.s.nc * a.s.H;
    const int logical = xcd_logical(blockIdx.x, n_wg);
    const int h = logical % a.s.H;
    const int c = (logical / a.s.H) % a.s.nc;
    const int b = logical / (a.s.H * a.s.nc);
    const int g = h / a.s.hpg;
    const int t0 = c * SQ;

    const int t = t0 + tid;
    const bool valid = t < a.s.L;
    const float dtv = a.dt[((size_t)b * a.s.L + min(t, a.s.L - 1)) * a.s.H + h];
    const float dtl = valid ? dtv : 0.f;
    const float a2 = block_scan(dtl * a.A[h], wsum) * LOG2E;
    a2s[tid] = a2;

    // stage x (256 rows x 8 chunks) and the entering state as bf16 (64 rows
    // x 16 chunks, each from 8 fp32)
    // this wave's 32-position blocks: {wave, 7 - wave} (balances the causal work)
    const int col = lane & 31, hl = lane >> 5;
    const int lbs[2] = {wave, 7 - wave};

    const size_t xrow = (size_t)a.s.H * SP;
#pragma unroll
    for (int i = 0; i < SQ * 8 / NT; ++i) {
        const int q = i * NT + tid, r = q >> 3, cc = q & 7;
        const int tr = min(t0 + r, a.s.L - 1);
        const u32x4 xv = ld_once<STREAM>(a.x + ((size_t)b * a.s.L + tr) * xrow + (size_t)h * SP + cc * 8);
        const u32x4 v = t0 + r < a.s.L ? xv : u32x4{0u, 0u, 0u, 0u};
        *(u32x4 *)(xt + r * (SP * 2) + ((cc ^ swz_tr128(r)) * 16)) = v;
    }
    const float *hin = a.prev + (((size_t)b * a.s.nc + c) * a.s.H + h) * (SP * SN);
#pragma unroll
    for (int i = 0; i < SP * 16 / NT; ++i) {
        const int q = i * NT + tid, r = q >> 4, cc = q & 15;
        const f32x4 f0 = ld_once<STREAM>(hin + r * SN + cc * 8);
        const f32x4 f1 = ld_once<STREAM>(hin + r * SN + cc * 8 + 4);
        const u32x4 v = {pack_bf16(f0[0], f0[1]), pack_bf16(f0[2], f0[3]), pack_bf16(f1[0], f1[1]),
                         pack_bf16(f1[2], f1[3])};
        *(u32x4 *)(ht + r * (SN * 2) + ((cc ^ swz_row256(r)) * 16)) = v;
    }
    __syncthreads();
    // The within-chunk weight exp(a_l - a_s) dt_s is split at the last
    // position e(s) of the 16-position block holding s:
    //   fs[s] = dt_s exp(a_e(s) - a_s)  (<= dt_s, formed once per position)
    //   r_l   = exp(a_l - a_e(s))       (one per lane and 16-position step)
    // so a weight costs two multiplies instead of an exponential.  Both
    // factors are finite for every (l, s) of a step: a_e - a_s spans at most
    // 16 positions; r_l > 1 only on steps crossing the diagonal, where the
    // products with s > l are masked to zero.
    fs[tid] = valid ? dtl * __builtin_amdgcn_exp2f(a2s[(tid | 15)] - a2) : 0.f;
    __syncthreads();

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][pb][r] = 0.f;

    // entering state: A = Hin rows (p), B = Cm rows (l), k = n.  A position
    // past L reads row L - 1: it only feeds an output row past L, which is
    // never stored.
    const size_t crow = (size_t)a.s.G * SN;
    const uint16_t *cp[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
        cp[i] = a.Cm + ((size_t)b * a.s.L + min(t0 + 32 * lbs[i] + col, a.s.L - 1)) * crow +
                (size_t)g * SN + 8 * hl;
#pragma unroll
    for (int ks = 0; ks < SN / 16; ++ks) {
        bf16x8 av[2];
#pragma unroll
        for (int pb = 0; pb < 2; ++pb) {
            const int r = 32 * pb + col;
            av[pb] = *(const bf16x8 *)(ht + r * (SN * 2) + (((2 * ks + hl) ^ swz_row256(r)) * 16));
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int pb = 0; pb < 2; ++pb)
                acc[i][pb] = mfma32(av[pb], __builtin_bit_cast(bf16x8, *(const u32x4 *)(cp[i] + 16 * ks)),
                                    acc[i][pb]);
    }
    // decay the entering state to each position (lane's column l)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const float e = exp2f(a2s[32 * lbs[i] + col]);
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[i][pb][r] *= e;
    }

    // within the chunk: A = x^T (p, s) by transpose reads, B = the weight
    // matrix M[l][s] = cb[l][s] exp(a_l - a_s) dt_s (s <= l).  M is built in
    // slabs of 32 positions s: all threads read the slab's cb rows (l >=
    // the slab start) with coalesced 16-byte loads, form the bf16 weights
    // and write them to an LDS tile (the entering state's space, free after
    // the first term); the waves then run the slab's two k-steps for their
    // own position blocks.  The cb loads of slab k + 1 are in flight during
    // the MFMAs of slab k.
    //   Weight of (l, s): cb[l][s] fs[s] r, with fs[s] = dt_s exp(a_e - a_s)
    // and r = exp(a_l - a_e) for e the last position of the 16-block of s
    // (one exponential per 4 weights; both factors finite, s > l masked).
    //   M tile: row l, 8-byte unit u (4 weights) at u ^ ((l >> 2) & 7), which
    // keeps both the staging writes and the operand reads conflict free.
    __syncthreads();   // every wave is done with the entering state
    unsigned char *mt = ht;
    const float *cbm = a.cb + (((size_t)b * a.s.nc + c) * a.s.G + g) * (SQ * SQ);
    const int ld_q = tid & 7;                  // 16-byte quad of the slab row
    float4 cr[8];                              // this thread's loads of one slab
    auto load_slab = [&](int k) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = 32 * k + (i * NT + tid) / 8;   // rows past 255 are not used
            if (i < 8 - k)
                cr[i] = *(const float4 *)(cbm + (size_t)row * SQ + 32 * k + 4 * ld_q);
        }
    };
    load_slab(0);
    for (int k = 0; k < SQ / 32; ++k) {
        // weights of slab k into the tile
        const int s0 = 32 * k + 4 * ld_q;
        const float4 fq = *(const float4 *)(fs + s0);
        const float a2e = a2s[(s0 | 15)];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (i < 8 - k) {
                const int row = 32 * k + (i * NT + tid) / 8;
                const float r = __builtin_amdgcn_exp2f(a2s[row] - a2e);
                const float4 cv4 = cr[i];
                const float w0 = s0 <= row ? cv4.x * fq.x * r : 0.f;
                const float w1 = s0 + 1 <= row ? cv4.y * fq.y * r : 0.f;
                const float w2 = s0 + 2 <= row ? cv4.z * fq.z * r : 0.f;
                const float w3 = s0 + 3 <= row ? cv4.w * fq.w * r : 0.f;
                *(u32x2 *)(mt + row * 64 + ((ld_q ^ ((row >> 2) & 7)) * 8)) =
                    u32x2{pack_bf16(w0, w1), pack_bf16(w2, w3)};
            }
        }
        __syncthreads();
        if (k + 1 < SQ / 32)
            load_slab(k + 1);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int lb = lbs[i];
            if (lb < k)
                continue;
            const int l = 32 * lb + col;
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const int u0 = 4 * kk + hl, u1 = u0 + 2;
                const u32x2 m0 = *(const u32x2 *)(mt + l * 64 + ((u0 ^ ((l >> 2) & 7)) * 8));
                const u32x2 m1 = *(const u32x2 *)(mt + l * 64 + ((u1 ^ ((l >> 2) & 7)) * 8));
                const bf16x8 bv = __builtin_bit_cast(bf16x8, u32x4{m0[0], m0[1], m1[0], m1[1]});
#pragma unroll
                for (int pb = 0; pb < 2; ++pb) {
                    const bf16x8 av =
                        tr_operand<SP * 2, swz_tr128>(xt, 32 * k + 16 * kk, 32 * pb, lane);
                    acc[i][pb] = mfma32(av, bv, acc[i][pb]);
                }
            }
        }
        __syncthreads();   // the tile is rewritten by the next slab
    }

    // skip term: lane holds y^T[p][l] for l = 32 lb + col and p = 32 pb +
    // 8 j + 4 hl + 0..3 (four consecutive p of output row l)
    const float dh = a.D ? a.D[h] : 0.f;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int l = 32 * lbs[i] + col;
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int p = 32 * pb + 8 * j + 4 * hl;
                const u32x2 xv = *(const u32x2 *)(xt + l * (SP * 2) + (((p >> 3) ^ swz_tr128(l)) * 16) +
                                                  (2 * p & 15));
                acc[i][pb][4 * j] += dh * bf16_lo(xv[0]);
                acc[i][pb][4 * j + 1] += dh * bf16_hi(xv[0]);
                acc[i][pb][4 * j + 2] += dh * bf16_lo(xv[1]);
                acc[i][pb][4 * j + 3] += dh * bf16_hi(xv[1]);
            }
    }
    // Store through LDS so that every global store writes whole rows: each
    // wave stages one 32 x 64 fp32 block at a time in its 8 KB of the x
    // tile (16-byte chunk q of row r at q ^ (r & 15), conflict free both
    // ways), then writes 4 rows of 256 bytes per instruction.  LDS accesses
    // of one wave complete in order, so the wave needs no barrier of its own.
    __syncthreads();   // every wave is done with the x tile
    float *stg = (float *)(xt + wave * (32 * SP * 4));
    const size_t xrow_ = (size_t)a.s.H * SP;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int pb = 0; pb < 2; ++pb)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int q = 8 * pb + 2 * j + hl;
                *(float4 *)(stg + col * SP + ((q ^ (col & 15)) * 4)) =
                    float4{acc[i][pb][4 * j], acc[i][pb][4 * j + 1], acc[i][pb][4 * j + 2],
                           acc[i][pb][4 * j + 3]};
            }
#pragma unroll
        for (int it = 0; it < 8; ++it) {
            const int r = 4 * it + (lane >> 4), q = lane & 15;
            const f32x4 v = *(const f32x4 *)(stg + r * SP + ((q ^ (r & 15)) * 4));
            const int tt = t0 + 32 * lbs[i] + r;
            if (tt < a.s.L)
                st_once<STREAM>(a.out + ((size_t)b * a.s.L + tt) * xrow_ + (size_t)h * SP + 4 * q, v);
        }
    }
}

// ---------------------------------------------------------------------------
// chunk matrix: cb^T[s][l] = sum_n Bm_s[n] Cm_l[n], eight waves, wave w owns
// the 32 rows s of block w and all 256 columns l

struct BmmArgs {
    SsdShape s;
    const uint16_t *Cm, *Bm;
    float *cb;
};

__global__ __launch_bounds__(512, 1) void bmm_chunk_kernel(BmmArgs args)
{
    const BmmArgs &a = args;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n_wg = a.s.B * a.s.nc * a.s.G;
    const int logical = xcd_logical(blockIdx.x, n_wg);
    const int g = logical % a.s.G;
    const int c = (logical / a.s.G) % a.s.nc;
    const int b = logical / (a.s.G * a.s.nc);
    const int t0 = c * SQ, col = lane & 31, hl = lane >> 5;
    const size_t row = (size_t)a.s.G * SN;
    f32x16 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc[j][r] = 0.f;
    const int ts = t0 + 32 * wave + col;
#pragma unroll 2
    for (int ks = 0; ks < SN / 16; ++ks) {
        const u32x4 va = load_row16(a.Bm + ((size_t)b * a.s.L + min(ts, a.s.L - 1)) * row +
                                        (size_t)g * SN + 16 * ks + 8 * hl,
                                    ts < a.s.L);
        const bf16x8 av = __builtin_bit_cast(bf16x8, va);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int tl = t0 + 32 * j + col;
            const u32x4 vb = load_row16(a.Cm + ((size_t)b * a.s.L + min(tl, a.s.L - 1)) * row +
                                            (size_t)g * SN + 16 * ks + 8 * hl,
                                        tl < a.s.L);
            acc[j] = mfma32(av, __builtin_bit_cast(bf16x8, vb), acc[j]);
        }
    }
    float *out = a.cb + (((size_t)b * a.s.nc + c) * a.s.G + g) * (SQ * SQ);
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int l = 32 * j + col, s = 32 * wave + 8 * q + 4 * hl;
            *(float4 *)(out + (size_t)l * SQ + s) =
                float4{acc[j][4 * q], acc[j][4 * q + 1], acc[j][4 * q + 2], acc[j][4 * q + 3]};
        }
}

// ---------------------------------------------------------------------------
// state passing: per (batch, head, quarter of the P x N state), sequential
// over chunks: prev[c] = H; H = exp(A sum_{l in c} dt_l) H + S_c

struct PassArgs {
    SsdShape s;
    const float *states, *dt, *A;
    float *prev, *final_states;
};

__global__ __launch_bounds__(NT, 4) void state_passing_kernel(PassArgs args)
{
    const PassArgs &a = args;
    __shared__ float wsum[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int qtr = blockIdx.x & 3;
    const int bh = blockIdx.x >> 2;
    const int h = bh % a.s.H, b = bh / a.s.H;
    const int e0 = qtr * (SP * SN / 4) + tid * 8;
    const float Ah = a.A[h];
    float4 h0 = {0.f, 0.f, 0.f, 0.f}, h1 = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < a.s.nc; ++c) {
        const int t = c * SQ + tid;
        const float dtv = a.dt[((size_t)b * a.s.L + min(t, a.s.L - 1)) * a.s.H + h];
        float v = t < a.s.L ? dtv : 0.f;
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1)
            v += __shfl_xor(v, d, 64);
        if (lane == 0)
            wsum[wave] = v;
        __syncthreads();
        const float decay = exp2f((wsum[0] + wsum[1] + wsum[2] + wsum[3]) * Ah * LOG2E);
        __syncthreads();
        const size_t off = (((size_t)b * a.s.nc + c) * a.s.H + h) * (SP * SN) + e0;
        *(float4 *)(a.prev + off) = h0;
        *(float4 *)(a.prev + off + 4) = h1;
        const float4 s0 = *(const float4 *)(a.states + off);
        const float4 s1 = *(const float4 *)(a.states + off + 4);
        h0 = float4{decay * h0.x + s0.x, decay * h0.y + s0.y, decay * h0.z + s0.z, decay * h0.w + s0.w};
        h1 = float4{decay * h1.x + s1.x, decay * h1.y + s1.y, decay * h1.z + s1.z, decay * h1.w + s1.w};
    }
    if (a.final_states) {
        float *f = a.final_states + ((size_t)b * a.s.H + h) * (SP * SN) + e0;
        *(float4 *)f = h0;
        *(float4 *)(f + 4) = h1;
    }
}

bool misaligned(const void *p) { return ((uintptr_t)p & 15u) != 0; }

bool overlaps(const void *p, size_t pn, const void *q, size_t qn)
{
    if (!p || !q)
        return false;
    const uintptr_t x = (uintptr_t)p, y = (uintptr_t)q;
    return x < y + qn && y < x + pn;
}

// shared shape validation; fills `s`
ta_status check_shape(int batch, int seqlen, int nheads, int ngroups, int headdim, int dstate,
                      int chunk_size, SsdShape &s)
{
    if (batch < 1 || seqlen < 1 || nheads < 1 || ngroups < 1 || nheads % ngroups)
        return TA_ERR_INVALID_SHAPE;
    if (headdim != SP || dstate != SN || chunk_size != SQ)
        return TA_ERR_UNSUPPORTED;
    const int64_t nc = ((int64_t)seqlen + SQ - 1) / SQ;
    // grid sizes and per-tensor element counts within the kernels' index types
    if ((int64_t)batch * nc * nheads >= (1ll << 31) || (int64_t)batch * nheads * 4 >= (1ll << 31) ||
        (int64_t)batch * nc * (nheads > ngroups ? nheads : ngroups) * SQ * SQ >= (1ll << 46))
        return TA_ERR_INVALID_SHAPE;
    s.B = batch;
    s.L = seqlen;
    s.H = nheads;
    s.G = ngroups;
    s.nc = (int)nc;
    s.hpg = nheads / ngroups;
    return TA_OK;
}

ta_status launched(hipError_t e) { return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH; }

}  // namespace

extern "C" {

ta_status ssd_chunk_state(const void *x, const void *Bm, const float *dt, const float *A,
                          float *states, int batch, int seqlen, int nheads, int ngroups,
                          int headdim, int dstate, int chunk_size, void *stream)
{
    if (!x || !Bm || !dt || !A || !states)
        return TA_ERR_NULL_POINTER;
    SsdShape s;
    const ta_status st = check_shape(batch, seqlen, nheads, ngroups, headdim, dstate, chunk_size, s);
    if (st != TA_OK)
        return st;
    if (misaligned(x) || misaligned(Bm) || misaligned(states) || ((uintptr_t)dt & 3) ||
        ((uintptr_t)A & 3))
        return TA_ERR_MISALIGNED;
    const size_t nx = (size_t)batch * seqlen * nheads * SP * 2, nb = (size_t)batch * seqlen * ngroups * SN * 2;
    const size_t ns = (size_t)batch * s.nc * nheads * SP * SN * 4;
    const size_t ndt = (size_t)batch * seqlen * nheads * 4;
    if (overlaps(states, ns, x, nx) || overlaps(states, ns, Bm, nb) || overlaps(states, ns, dt, ndt) ||
        overlaps(states, ns, A, (size_t)nheads * 4))
        return TA_ERR_ALIASING;
    StateArgs a{s, (const uint16_t *)x, (const uint16_t *)Bm, dt, A, states};
    // two heads per workgroup when a group holds an even number of heads and
    // the grid keeps at least four workgroups per CU (smaller grids run
    // faster with one head each: B=1 L=2048 2.85 against 3.12 TB/s)
    const bool strm = nx + ns > STREAM_BYTES;
    const hipStream_t hs = (hipStream_t)stream;
    if (s.hpg % 2 == 0 && (int64_t)s.B * s.nc * (s.H / 2) >= 1024) {
        const dim3 grid(s.B * s.nc * (s.H / 2));
        if (strm)
            hipLaunchKernelGGL((chunk_state_kernel<2, true>), grid, dim3(NT), 0, hs, a);
        else
            hipLaunchKernelGGL((chunk_state_kernel<2, false>), grid, dim3(NT), 0, hs, a);
    } else {
        const dim3 grid(s.B * s.nc * s.H);
        if (strm)
            hipLaunchKernelGGL((chunk_state_kernel<1, true>), grid, dim3(NT), 0, hs, a);
        else
            hipLaunchKernelGGL((chunk_state_kernel<1, false>), grid, dim3(NT), 0, hs, a);
    }
    return launched(hipGetLastError());
}

ta_status ssd_chunk_scan(const void *x, const void *Cm, const float *cb, const float *dt,
                         const float *A, const float *prev_states, const float *D, float *out,
                         int batch, int seqlen, int nheads, int ngroups, int headdim, int dstate,
                         int chunk_size, void *stream)
{
    if (!x || !Cm || !cb || !dt || !A || !prev_states || !out)
        return TA_ERR_NULL_POINTER;
    SsdShape s;
    const ta_status st = check_shape(batch, seqlen, nheads, ngroups, headdim, dstate, chunk_size, s);
    if (st != TA_OK)
        return st;
    if (misaligned(x) || misaligned(Cm) || misaligned(cb) || misaligned(prev_states) ||
        misaligned(out) || ((uintptr_t)dt & 3) || ((uintptr_t)A & 3) || ((uintptr_t)D & 3))
        return TA_ERR_MISALIGNED;
    const size_t nx = (size_t)batch * seqlen * nheads * SP;
    const size_t no = nx * 4;
    const size_t ins[][2] = {
        {(size_t)x, nx * 2},
        {(size_t)Cm, (size_t)batch * seqlen * ngroups * SN * 2},
        {(size_t)cb, (size_t)batch * s.nc * ngroups * SQ * SQ * 4},
        {(size_t)dt, (size_t)batch * seqlen * nheads * 4},
        {(size_t)A, (size_t)nheads * 4},
        {(size_t)prev_states, (size_t)batch * s.nc * nheads * SP * SN * 4},
        {(size_t)D, D ? (size_t)nheads * 4 : 0},
    };
    for (const auto &in : ins)
        if (overlaps(out, no, (const void *)in[0], in[1]))
            return TA_ERR_ALIASING;
    ScanArgs a{s, (const uint16_t *)x, (const uint16_t *)Cm, cb, dt, A, prev_states, D, out};
    // x, the entering states and y: the streams read or written once
    if (nx * 2 + ins[5][1] + no > STREAM_BYTES)
        hipLaunchKernelGGL(chunk_scan_kernel<true>, dim3(s.B * s.nc * s.H), dim3(NT), 0,
                           (hipStream_t)stream, a);
    else
        hipLaunchKernelGGL(chunk_scan_kernel<false>, dim3(s.B * s.nc * s.H), dim3(NT), 0,
                           (hipStream_t)stream, a);
    return launched(hipGetLastError());
}

ta_status ssd_bmm_chunk(const void *Cm, const void *Bm, float *cb, int batch, int seqlen,
                        int ngroups, int dstate, int chunk_size, void *stream)
{
    if (!Cm || !Bm || !cb)
        return TA_ERR_NULL_POINTER;
    SsdShape s;
    const ta_status st = check_shape(batch, seqlen, ngroups, ngroups, SP, dstate, chunk_size, s);
    if (st != TA_OK)
        return st;
    if (misaligned(Cm) || misaligned(Bm) || misaligned(cb))
        return TA_ERR_MISALIGNED;
    const size_t nbc = (size_t)batch * seqlen * ngroups * SN * 2;
    const size_t ncb = (size_t)batch * s.nc * ngroups * SQ * SQ * 4;
    if (overlaps(cb, ncb, Cm, nbc) || overlaps(cb, ncb, Bm, nbc))
        return TA_ERR_ALIASING;
    BmmArgs a{s, (const uint16_t *)Cm, (const uint16_t *)Bm, cb};
    hipLaunchKernelGGL(bmm_chunk_kernel, dim3(s.B * s.nc * s.G), dim3(512), 0, (hipStream_t)stream, a);
    return launched(hipGetLastError());
}

ta_status ssd_state_passing(const float *states, const float *dt, const float *A, float *prev_states,
                            float *final_states, int batch, int seqlen, int nheads, int headdim,
                            int dstate, int chunk_size, void *stream)
{
    if (!states || !dt || !A || !prev_states)
        return TA_ERR_NULL_POINTER;
    SsdShape s;
    const ta_status st = check_shape(batch, seqlen, nheads, 1, headdim, dstate, chunk_size, s);
    if (st != TA_OK)
        return st;
    if (misaligned(states) || misaligned(prev_states) || misaligned(final_states) ||
        ((uintptr_t)dt & 3) || ((uintptr_t)A & 3))
        return TA_ERR_MISALIGNED;
    const size_t ns = (size_t)batch * s.nc * nheads * SP * SN * 4;
    const size_t nf = (size_t)batch * nheads * SP * SN * 4;
    const size_t ndt = (size_t)batch * seqlen * nheads * 4;
    if (overlaps(prev_states, ns, states, ns) || overlaps(prev_states, ns, dt, ndt) ||
        overlaps(prev_states, ns, A, (size_t)nheads * 4) || overlaps(final_states, nf, states, ns) ||
        overlaps(final_states, nf, prev_states, ns) || overlaps(final_states, nf, dt, ndt) ||
        overlaps(final_states, nf, A, (size_t)nheads * 4))
        return TA_ERR_ALIASING;
    PassArgs a{s, states, dt, A, prev_states, final_states};
    hipLaunchKernelGGL(state_passing_kernel, dim3(s.B * s.H * 4), dim3(NT), 0, (hipStream_t)stream, a);
    return launched(hipGetLastError());
}

}  // extern "C"
