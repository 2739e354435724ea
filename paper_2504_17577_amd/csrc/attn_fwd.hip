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
//    query l % 32, so every row reduction is in-lane plus one exchange with
//    lane l ^ 32.
//  * The same lane ownership carries into O^T = V^T P^T: the exponentials
//    of the scores, rounded to bf16, already sit in the B-operand layout
//    (query = lane % 32); the reduction order of the 16 keys per MFMA step
//    is chosen to match that, and V is stored transposed in LDS with the
//    same key order so each A operand is one 16-byte LDS read.
//  * The per-row rescale factor is then a per-lane scalar.
//  * K and V^T tiles are double-buffered in LDS: the global loads of tile
//    j+1 are issued before the math on tile j and written to the other
//    buffer after it, with one barrier per tile.  16-byte LDS chunks are
//    XOR-swizzled by row so the MFMA operand reads are conflict-free.
//  * Causal: key tiles beyond the last visible key of the workgroup are not
//    visited; only tiles crossing the diagonal or the end of the sequence
//    take the masked path; waves whose queries see none of a tile skip it.
//  * Grid: one workgroup per (batch, head, query tile); consecutive workgroup
//    ids are spread over the 8 XCDs by the hardware, so ids are remapped to
//    give each XCD a contiguous range of heads (their K/V stay in that XCD's
//    L2), heaviest causal tiles first.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tileattn.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128;      // query rows per workgroup (4 waves x 32)
constexpr int BN = 64;       // keys per tile
constexpr int NT = 256;      // threads per workgroup
constexpr int NXCD = 8;      // XCDs per MI355X
constexpr float LOG2E = 1.44269504088896340736f;
constexpr float LN2 = 0.69314718055994530942f;

template <int D>
struct Cfg {
    static constexpr int CH = D / 8;                        // 16-byte chunks per K row
    static constexpr int K_BYTES = BN * D * 2;              // K tile [BN][D]
    static constexpr int V_BYTES = D * BN * 2;              // V^T tile [D][BN]
    static constexpr int STAGE = K_BYTES + V_BYTES;
    static constexpr int K_LOADS = BN * CH / NT;            // 16-byte K loads / thread / tile
    static constexpr int V_UNITS = (BN / 8) * (D / 2) / NT; // 8-key x 2-d V units / thread
    static constexpr int DB = D / 32;                       // 32-row blocks of O^T
    static constexpr int KK = D / 16;                       // MFMA k-steps for S^T
    static_assert(BN * CH % NT == 0 && (BN / 8) * (D / 2) % NT == 0, "tile/thread mismatch");
};

struct Args {
    const uint16_t *Q, *K, *V;
    float *O, *LSE;
    int B, Hq, Hkv, Sq, Sk;
    int group;       // Hq / Hkv
    int n_qt;        // query tiles per head
    int n_wg;        // total workgroups
    float c;         // scale * log2(e)
};

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    __bf16 a = (__bf16)lo, b = (__bf16)hi;   // round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, a) |
           ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Workgroup id -> (head index b*Hq+h, query tile).  The hardware hands
// workgroup i to XCD i % 8; give each XCD a contiguous block of logical ids.
__device__ __forceinline__ void decode_wg(const Args &a, int bid, int &head, int &qt)
{
    const int per = a.n_wg / NXCD, rem = a.n_wg % NXCD;
    const int xcd = bid % NXCD, idx = bid / NXCD;
    const int logical = xcd * per + (xcd < rem ? xcd : rem) + idx;
    head = logical / a.n_qt;
    qt = logical % a.n_qt;
}

template <int D, bool CAUSAL>
__global__ __launch_bounds__(NT, 2) void attn_fwd_kernel(Args a)
{
    using C = Cfg<D>;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int col = lane & 31, half = lane >> 5;

    int head, qt;
    decode_wg(a, blockIdx.x, head, qt);
    if (CAUSAL)
        qt = a.n_qt - 1 - qt;   // heaviest query tiles of a head first
    const int b = head / a.Hq, hq = head % a.Hq;
    const int hk = hq / a.group;
    const int off = a.Sk - a.Sq;  // bottom-right causal offset

    const int q0 = qt * BM;
    const int qi = q0 + wave * 32 + col;             // this lane's query row
    const int q_last_wg = min(q0 + BM, a.Sq) - 1;    // last real query of the workgroup
    const int q_last_wave = min(q0 + wave * 32 + 31, a.Sq - 1);

    // key tiles to visit, and the first one needing per-element masks
    const int n_kv_all = (a.Sk + BN - 1) / BN;
    int n_kv = n_kv_all;
    int first_masked = (a.Sk % BN) ? n_kv_all - 1 : n_kv_all;
    if (CAUSAL) {
        n_kv = min(n_kv_all, (q_last_wg + off) / BN + 1);
        // tile j needs masks if its last key exceeds what the first query sees
        first_masked = min(first_masked, max(0, (q0 + off + 1) / BN));
        first_masked = min(first_masked, n_kv);
    }

    const size_t kv_base = ((size_t)b * a.Hkv + hk) * (size_t)a.Sk * D;
    const uint16_t *Kg = a.K + kv_base;
    const uint16_t *Vg = a.V + kv_base;

    // ---- Q for this lane's query, as the B operand of S^T = K Q^T --------
    bf16x8 qreg[C::KK];
    {
        const uint16_t *qp = a.Q + (((size_t)b * a.Hq + hq) * a.Sq + qi) * D + 8 * half;
#pragma unroll
        for (int kk = 0; kk < C::KK; ++kk) {
            u32x4 v = {0u, 0u, 0u, 0u};
            if (qi < a.Sq)
                v = *(const u32x4 *)(qp + 16 * kk);
            qreg[kk] = __builtin_bit_cast(bf16x8, v);
        }
    }

    // ---- tile staging: global -> registers -> LDS -------------------------
    u32x4 kst[C::K_LOADS];
    uint32_t vst[C::V_UNITS][8];

    auto load_tile = [&](int j) {
#pragma unroll
        for (int i = 0; i < C::K_LOADS; ++i) {
            const int id = tid + NT * i;
            const int row = id / C::CH, ch = id % C::CH;
            const int key = j * BN + row;
            u32x4 v = {0u, 0u, 0u, 0u};
            if (key < a.Sk)
                v = *(const u32x4 *)(Kg + (size_t)key * D + 8 * ch);
            kst[i] = v;
        }
#pragma unroll
        for (int i = 0; i < C::V_UNITS; ++i) {
            const int u = tid + NT * i;
            const int dp = u % (D / 2), cu = u / (D / 2);
            const int kbase = j * BN + 16 * (cu >> 1) + 4 * (cu & 1);
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int key = kbase + (t & 3) + 8 * (t >> 2);
                uint32_t v = 0u;
                if (key < a.Sk)
                    v = *(const uint32_t *)(Vg + (size_t)key * D + 2 * dp);
                vst[i][t] = v;
            }
        }
    };

    auto store_tile = [&](int stage) {
        unsigned char *ks = smem + stage * C::STAGE;
        unsigned char *vs = ks + C::K_BYTES;
#pragma unroll
        for (int i = 0; i < C::K_LOADS; ++i) {
            const int id = tid + NT * i;
            const int row = id / C::CH, ch = id % C::CH;
            *(u32x4 *)(ks + row * (D * 2) + ((ch ^ (row & (C::CH - 1))) * 16)) = kst[i];
        }
#pragma unroll
        for (int i = 0; i < C::V_UNITS; ++i) {
            const int u = tid + NT * i;
            const int dp = u % (D / 2), cu = u / (D / 2);
            u32x4 lo, hi;   // rows d = 2dp and 2dp+1 of V^T, 8 keys each
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const uint32_t x0 = vst[i][2 * t], x1 = vst[i][2 * t + 1];
                lo[t] = (x0 & 0xFFFFu) | (x1 << 16);
                hi[t] = (x0 >> 16) | (x1 & 0xFFFF0000u);
            }
            const int d0 = 2 * dp, d1 = 2 * dp + 1;
            *(u32x4 *)(vs + d0 * (BN * 2) + ((cu ^ (d0 & 7)) * 16)) = lo;
            *(u32x4 *)(vs + d1 * (BN * 2) + ((cu ^ (d1 & 7)) * 16)) = hi;
        }
    };

    // ---- softmax state and accumulator -------------------------------------
    f32x16 acc_o[C::DB];
#pragma unroll
    for (int db = 0; db < C::DB; ++db)
        for (int r = 0; r < 16; ++r)
            acc_o[db][r] = 0.f;
    float m_run = -INFINITY;   // running max of scale*log2(e)*s (same in both halves)
    float l_run = 0.f;         // running sum of this half's keys

    if (n_kv > 0) {
        load_tile(0);
        store_tile(0);
    }
    __syncthreads();

    for (int j = 0; j < n_kv; ++j) {
        const int stage = j & 1;
        const bool more = j + 1 < n_kv;
        if (more)
            load_tile(j + 1);

        const unsigned char *ks = smem + stage * C::STAGE;
        const unsigned char *vs = ks + C::K_BYTES;
        const bool wave_active =
            (q0 + wave * 32 < a.Sq) && (!CAUSAL || j * BN <= q_last_wave + off);

        if (wave_active) {
            // S^T[key][query] for the two 32-key blocks of this tile
            f32x16 s[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                for (int r = 0; r < 16; ++r)
                    s[kb][r] = 0.f;
                const int row = 32 * kb + col;
                const unsigned char *kr = ks + row * (D * 2);
#pragma unroll
                for (int kk = 0; kk < C::KK; ++kk) {
                    const int ch = (2 * kk + half) ^ (row & (C::CH - 1));
                    const bf16x8 av = *(const bf16x8 *)(kr + ch * 16);
                    s[kb] = mfma32(av, qreg[kk], s[kb]);
                }
            }

            // lane holds keys 32kb + 8(r/4) + 4half + r%4 of query qi
            const bool masked = j >= first_masked;
            float mx = -INFINITY;
            if (masked) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = j * BN + 32 * kb + 8 * (r >> 2) + 4 * half + (r & 3);
                        const bool ok = key < a.Sk && (!CAUSAL || key <= qi + off);
                        if (!ok)
                            s[kb][r] = -INFINITY;
                        mx = fmaxf(mx, s[kb][r]);
                    }
            } else {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        mx = fmaxf(mx, s[kb][r]);
            }
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            // new running max in the base-2 domain; -inf while nothing is visible
            const float m_tile = (mx == -INFINITY) ? -INFINITY : mx * a.c;
            const float m_new = fmaxf(m_run, m_tile);
            const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
            m_run = m_new;

            float rowsum = 0.f;
            uint32_t pk[2][8];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int r = 0; r < 16; r += 2) {
                    float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][r], a.c, -m_use));
                    float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][r + 1], a.c, -m_use));
                    if (masked) {
                        p0 = (s[kb][r] == -INFINITY) ? 0.f : p0;
                        p1 = (s[kb][r + 1] == -INFINITY) ? 0.f : p1;
                    }
                    rowsum += p0 + p1;
                    pk[kb][r >> 1] = pack_bf16(p0, p1);
                }
            l_run = l_run * alpha + rowsum;

#pragma unroll
            for (int db = 0; db < C::DB; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc_o[db][r] *= alpha;

            // O^T[d][query] += V^T[d][key] P^T[key][query], 16 keys per step:
            // k-step ks uses keys 16ks + {4half..4half+3, 8+4half..8+4half+3}
#pragma unroll
            for (int ks2 = 0; ks2 < BN / 16; ++ks2) {
                const int kb = ks2 >> 1, rb = (ks2 & 1) * 4;
                u32x4 bw = {pk[kb][rb], pk[kb][rb + 1], pk[kb][rb + 2], pk[kb][rb + 3]};
                const bf16x8 bv = __builtin_bit_cast(bf16x8, bw);
#pragma unroll
                for (int db = 0; db < C::DB; ++db) {
                    const int d = 32 * db + col;
                    const int ch = (2 * ks2 + half) ^ (d & 7);
                    const bf16x8 av = *(const bf16x8 *)(vs + d * (BN * 2) + ch * 16);
                    acc_o[db] = mfma32(av, bv, acc_o[db]);
                }
            }
        }

        if (more)
            store_tile(stage ^ 1);
        __syncthreads();
    }

    // ---- epilogue: normalise, store O rows and LSE ------------------------
    const float l = l_run + __shfl_xor(l_run, 32);
    if (qi < a.Sq) {
        const float inv = 1.f / l;
        float *op = a.O + (((size_t)b * a.Hq + hq) * a.Sq + qi) * D;
#pragma unroll
        for (int db = 0; db < C::DB; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                float4 v;
                v.x = acc_o[db][4 * g + 0] * inv;
                v.y = acc_o[db][4 * g + 1] * inv;
                v.z = acc_o[db][4 * g + 2] * inv;
                v.w = acc_o[db][4 * g + 3] * inv;
                *(float4 *)(op + 32 * db + 8 * g + 4 * half) = v;
            }
        if (half == 0)
            a.LSE[((size_t)b * a.Hq + hq) * a.Sq + qi] = (m_run + log2f(l)) * LN2;
    }
}

template <int D, bool CAUSAL>
hipError_t launch(const Args &a, hipStream_t stream)
{
    constexpr int lds = 2 * Cfg<D>::STAGE;
    hipLaunchKernelGGL((attn_fwd_kernel<D, CAUSAL>), dim3(a.n_wg), dim3(NT), lds, stream, a);
    return hipGetLastError();
}

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

}  // namespace

extern "C" {

ta_status attn_fwd(const void *Q, const void *K, const void *V, float *O, float *LSE, int B,
                   int Hq, int Hkv, int Sq, int Sk, int D, int causal, float scale, void *stream)
{
    if (!Q || !K || !V || !O || !LSE)
        return TA_ERR_NULL_POINTER;
    if (B < 1 || Hq < 1 || Hkv < 1 || Sq < 1 || Sk < 1 || D < 1)
        return TA_ERR_INVALID_SHAPE;
    if (Hq % Hkv != 0 || (causal && Sq > Sk))
        return TA_ERR_INVALID_SHAPE;
    if (D != 64 && D != 128)
        return TA_ERR_UNSUPPORTED;
    // 32-bit in-kernel offsets are used within one (batch, head) slice only;
    // the grid itself must fit a 32-bit workgroup count
    const int64_t n_qt = ((int64_t)Sq + BM - 1) / BM;
    const int64_t n_wg = (int64_t)B * Hq * n_qt;
    if ((int64_t)Sq * D >= (1ll << 31) || (int64_t)Sk * D >= (1ll << 31) || n_wg >= (1ll << 31))
        return TA_ERR_INVALID_SHAPE;
    if (misaligned(Q) || misaligned(K) || misaligned(V) || misaligned(O) || misaligned(LSE))
        return TA_ERR_MISALIGNED;
    if (!(scale >= 0.f) || !isfinite(scale))
        return TA_ERR_INVALID_SCALE;
    const size_t nq = (size_t)B * Hq * Sq * D, nkv = (size_t)B * Hkv * Sk * D;
    const size_t nl = (size_t)B * Hq * Sq;
    const size_t o_bytes = nq * 4, l_bytes = nl * 4;
    if (overlaps(O, o_bytes, Q, nq * 2) || overlaps(O, o_bytes, K, nkv * 2) ||
        overlaps(O, o_bytes, V, nkv * 2) || overlaps(LSE, l_bytes, Q, nq * 2) ||
        overlaps(LSE, l_bytes, K, nkv * 2) || overlaps(LSE, l_bytes, V, nkv * 2) ||
        overlaps(O, o_bytes, LSE, l_bytes))
        return TA_ERR_ALIASING;

    Args a;
    a.Q = (const uint16_t *)Q;
    a.K = (const uint16_t *)K;
    a.V = (const uint16_t *)V;
    a.O = O;
    a.LSE = LSE;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.Sq = Sq;
    a.Sk = Sk;
    a.group = Hq / Hkv;
    a.n_qt = (int)n_qt;
    a.n_wg = (int)n_wg;
    a.c = scale * LOG2E;

    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (D == 64)
        e = causal ? launch<64, true>(a, s) : launch<64, false>(a, s);
    else
        e = causal ? launch<128, true>(a, s) : launch<128, false>(a, s);
    return e == hipSuccess ? TA_OK : TA_ERR_LAUNCH;
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
    }
    return "unknown status";
}

int ta_version(void) { return 100; }

}  // extern "C"
