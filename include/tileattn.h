/*
 * tileattn — fused scaled-dot-product attention forward for AMD MI355X
 * (gfx950), as a C ABI.
 *
 * The operation is the tile-fused attention kernel of the TileLang paper
 * (arXiv 2504.17577): scores S = scale * Q K^T, a softmax over keys computed
 * online over key tiles (running row max, rescale of the partial sums by the
 * exponential of the max difference, running row sum, final division), and
 * O = softmax(S) V, without ever storing S in memory.  The paper prints this
 * recurrence in its appendix listing "Implementation of FlashMLA with
 * TileLang" and benchmarks the multi-head forward in its FlashAttention
 * experiment (Section "Numerical Experiments", table "FlashAttention shapes
 * in our benchmark": batch, heads, sequence length, head dim 128, causal).
 *
 * Conventions for every entry point below:
 *   - Layouts are contiguous row-major BHSD: Q and O are [B, Hq, Sq, D],
 *     K and V are [B, Hkv, Sk, D], LSE is [B, Hq, Sq].  There are no stride
 *     arguments.
 *   - The caller owns every buffer.  The library allocates nothing, frees
 *     nothing and keeps no state between calls; calls are thread-safe.
 *   - Calls are asynchronous: they validate, enqueue on `stream` and return.
 *     `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - All validation happens before any HIP call: a status other than TA_OK
 *     means nothing was enqueued and no HIP API was touched (except for
 *     TA_ERR_LAUNCH, reported by the HIP runtime after the launch).
 *   - O and LSE are fully overwritten, never accumulated into.
 */
#ifndef TILEATTN_H
#define TILEATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TA_OK = 0,
    TA_ERR_NULL_POINTER = 1,  /* a required pointer is NULL                                 */
    TA_ERR_INVALID_SHAPE = 2, /* a size < 1, Hq % Hkv != 0, causal with Sq > Sk, or an
                                 element count beyond 2^31 per (batch, head) slice         */
    TA_ERR_UNSUPPORTED = 3,   /* D is not 64 or 128                                         */
    TA_ERR_MISALIGNED = 4,    /* a pointer is not 16-byte aligned                           */
    TA_ERR_INVALID_SCALE = 5, /* scale is negative, NaN or infinite                         */
    TA_ERR_ALIASING = 6,      /* O or LSE overlaps an input or each other                   */
    TA_ERR_LAUNCH = 7,        /* the HIP runtime reported an error for the launch           */
    TA_ERR_WORKSPACE = 8,     /* attn_fwd_split: workspace NULL or smaller than required    */
    TA_ERR_SCRATCH = 9        /* attn_fwd_split_noalloc: partial results larger than
                                 TA_SPLIT_SCRATCH_BYTES                                    */
} ta_status;

/*
 * attn_fwd — O = softmax(scale * Q K^T [+ causal mask]) V and its row
 * log-sum-exp, for bf16 inputs with fp32 accumulation.
 *
 *   Q    device, bf16 [B, Hq, Sq, D]           read only
 *   K    device, bf16 [B, Hkv, Sk, D]          read only
 *   V    device, bf16 [B, Hkv, Sk, D]          read only
 *   O    device, fp32 [B, Hq, Sq, D]           written
 *   LSE  device, fp32 [B, Hq, Sq]              written: natural log of
 *        sum_j exp(scale * q_i . k_j) over the keys row i may see
 *   Hq % Hkv == 0; query head h reads key/value head h / (Hq / Hkv)
 *   causal != 0: key j is visible to query i iff j <= i + (Sk - Sq)
 *        (bottom-right alignment; requires Sq <= Sk so every row sees a key)
 *   scale >= 0, finite; the kernel works in base 2 internally
 *   D in {64, 128}; every pointer 16-byte aligned
 *   stream: hipStream_t as void*
 *
 * The scores are formed in fp32 from bf16 products; the softmax weights are
 * rounded to bf16 (round to nearest even) before the P V product.
 */
ta_status attn_fwd(const void *Q, const void *K, const void *V, float *O, float *LSE,
                   int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal, float scale,
                   void *stream);

/*
 * attn_fwd_bf16out — attn_fwd with O written in bf16 instead of fp32.
 *
 *   O    device, bf16 [B, Hq, Sq, D]           written: each element is the
 *        fp32 value attn_fwd would store, rounded to nearest even
 *   every other argument, the validation and the status codes as attn_fwd;
 *   the aliasing check uses the bf16 size of O
 *
 * For callers that keep activations in bf16 (the usual next consumer of an
 * attention output is a bf16 projection); halves the output traffic.
 */
ta_status attn_fwd_bf16out(const void *Q, const void *K, const void *V, void *O, float *LSE,
                           int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                           float scale, void *stream);

/*
 * attn_fwd_split — attn_fwd with the key range of every query tile split
 * over `num_splits` workgroups, for grids too small to fill the GPU (few
 * heads, short query blocks against long key sequences).
 *
 * Each split computes the softmax result of its rows over its own keys,
 * (O_s, LSE_s), into the workspace; a second kernel merges them exactly:
 * LSE = log sum_s exp(LSE_s) and O = sum_s exp(LSE_s - LSE) O_s.  This is the
 * same rescaling the online softmax applies between key tiles, applied
 * between splits.  Results agree with attn_fwd to within fp32 rounding.
 *
 *   O          device, [B, Hq, Sq, D]: fp32, or bf16 if o_bf16 != 0
 *   num_splits 1..128 requested; splits are whole key tiles, so at most
 *              ceil(Sk / BN) are launched; 1 runs attn_fwd / attn_fwd_bf16out
 *              and ignores the workspace
 *   workspace  device, 16-byte aligned, at least the size
 *              ta_split_workspace_bytes reports (owned by the caller, which
 *              may reuse it once the call's work on `stream` has finished;
 *              its contents on entry do not matter); must not overlap any
 *              other argument (TA_ERR_ALIASING)
 *   other arguments, validation and status codes as attn_fwd;
 *   TA_ERR_WORKSPACE if num_splits > 1 and workspace is NULL or too small
 */
ta_status attn_fwd_split(const void *Q, const void *K, const void *V, void *O, int o_bf16,
                         float *LSE, int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                         float scale, int num_splits, void *workspace, size_t workspace_bytes,
                         void *stream);

/*
 * attn_fwd_split_noalloc — attn_fwd_split for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  The per-split partial results go to a
 * static device array inside the library (TA_SPLIT_SCRATCH_BYTES per GPU,
 * allocated when the library's code is loaded on that GPU and held until the
 * process ends) instead of a caller workspace; the call itself allocates and
 * frees nothing.
 *
 *   arguments, results and status codes as attn_fwd_split without the
 *   workspace; TA_ERR_SCRATCH (before any HIP call) if the partial results,
 *   num_splits' * B*Hq*Sq * (D + 1) * 4 bytes for the num_splits' splits
 *   actually launched, exceed TA_SPLIT_SCRATCH_BYTES; num_splits == 1 runs
 *   attn_fwd / attn_fwd_bf16out and touches no scratch.
 *   TA_ERR_LAUNCH also if the runtime cannot report the current device or
 *   the scratch's address on it (looked up once per device, on the first
 *   call there, with that device current).
 *
 * Every call on one GPU uses that GPU's one scratch array: calls whose work
 * overlaps on one GPU (different streams, or different host threads without
 * ordering) race on it and give wrong results.  Calls ordered on one stream
 * are safe.  The scratch keeps the last call's contents; nothing in it needs
 * clearing, since every launched split writes all of its partial rows before
 * the merge reads them.
 */
#define TA_SPLIT_SCRATCH_BYTES (64ull << 20)
ta_status attn_fwd_split_noalloc(const void *Q, const void *K, const void *V, void *O,
                                 int o_bf16, float *LSE, int B, int Hq, int Hkv, int Sq, int Sk,
                                 int D, int causal, float scale, int num_splits, void *stream);

/* Workspace bytes attn_fwd_split needs: num_splits * B*Hq*Sq * (D + 1) * 4
 * for num_splits > 1 (fp32 partial O and LSE per split), 0 for 1.
 * TA_ERR_INVALID_SHAPE / TA_ERR_UNSUPPORTED / TA_ERR_NULL_POINTER as above.
 * No HIP call. */
ta_status ta_split_workspace_bytes(int B, int Hq, int Sq, int D, int num_splits,
                                   size_t *bytes);

/* A split count for attn_fwd_split: 1 when B*Hq*ceil(Sq/BM) workgroups
 * already give two per CU (512), else enough splits to reach that, keeping
 * at least 32 key tiles (2048 keys) per split: shorter splits lose more to
 * the merge kernel's launch and traffic than the extra workgroups win.
 * No HIP call. */
ta_status ta_split_heuristic(int B, int Hq, int Hkv, int Sq, int Sk, int D, int causal,
                             int *num_splits);

/*
 * mla_decode — multi-head latent attention, one decode step: the
 * computation of the paper's appendix listing "Implementation of FlashMLA
 * with TileLang".  For batch b and query head h, with latent head
 * hk = h / (H / Hkv), over all Skv cache positions t:
 *   s_t = scale * (Q[b,h,:] . KV[b,t,hk,:] + Q_pe[b,h,:] . K_pe[b,t,hk,:])
 *   O[b,h,:] = sum_t softmax(s)_t KV[b,t,hk,:]      (the latent cache is the value)
 *   LSE[b,h] = ln sum_t exp(s_t)
 *
 *   Q     device, bf16 [B, H, Dl]             read only
 *   Q_pe  device, bf16 [B, H, Dr]             read only
 *   KV    device, bf16 [B, Skv, Hkv, Dl]      read only (the listing's layout)
 *   K_pe  device, bf16 [B, Skv, Hkv, Dr]      read only
 *   O     device, fp32 [B, H, Dl]             written
 *   LSE   device, fp32 [B, H]                 written (natural log, scale included)
 *   Dl == 512 and Dr == 64 (else TA_ERR_UNSUPPORTED); H % Hkv == 0
 *   num_splits: 1..128 requested splits of the cache positions (whole tiles
 *   of 32; trailing empty splits are dropped); for more than one, the
 *   per-split results go to `workspace` (device, 16-byte aligned, at least
 *   mla_workspace_bytes(B, H, num_splits) bytes, owned by the caller, no
 *   overlap with any other argument) and a second kernel merges them;
 *   num_splits == 1 ignores the workspace
 *   scale >= 0, finite; every pointer 16-byte aligned; stream as attn_fwd
 * Status codes as attn_fwd (TA_ERR_WORKSPACE for a missing or small
 * workspace).  Scores and sums are fp32, the softmax weights bf16 for the
 * weighted sum of the latent rows.
 */
ta_status mla_decode(const void *Q, const void *Q_pe, const void *KV, const void *K_pe,
                     float *O, float *LSE, int B, int H, int Hkv, int Skv, int Dl, int Dr,
                     float scale, int num_splits, void *workspace, size_t workspace_bytes,
                     void *stream);

/* Workspace bytes mla_decode needs: num_splits * B*H * (Dl + 1) * 4 with
 * Dl = 512 for num_splits > 1, 0 for 1.  No HIP call. */
ta_status mla_workspace_bytes(int B, int H, int num_splits, size_t *bytes);

/* A split count for mla_decode: enough splits of the cache for one
 * workgroup per CU (a workgroup covers 128 query heads of one latent head and
 * fills its CU's registers), keeping at least 8 tiles (256 positions) per
 * split.  No HIP call. */
ta_status mla_split_heuristic(int B, int H, int Hkv, int Skv, int *num_splits);

/*
 * gemm_bf16 — C = A B: the kernel beneath the paper's Matmul listing
 * (appendix "Matrix Multiplication (Matmul)"), bf16 inputs, fp32
 * accumulation.
 *
 *   A  device, bf16 [M, K] row-major         read only
 *   B  device, bf16 [K, N] row-major         read only
 *   C  device, [M, N] row-major: fp32, or bf16 (rounded to nearest even) if
 *      c_bf16 != 0                             written
 *   M % 128 == 0, N % 128 == 0, K % 64 == 0, and K * N * 2 < 2^31 (else
 *   TA_ERR_UNSUPPORTED, resp. TA_ERR_INVALID_SHAPE for the size); or M == 1,
 *   the matrix-vector product of the paper's V0-V7 shapes (appendix table
 *   "Matrix shapes in our benchmark"), with N % 64 == 0 and K % 8 == 0, which
 *   runs a separate HBM-bound kernel on the vector ALUs; every pointer
 *   16-byte aligned; C must not overlap A or B; stream as attn_fwd.
 * Status codes as attn_fwd; validation before any HIP call.
 */
ta_status gemm_bf16(const void *A, const void *B, void *C, int c_bf16, int M, int N, int K,
                    void *stream);

/*
 * gemv_bf16_split — the matrix-vector product C[n] = sum_k A[k] B[k][n] of
 * gemm_bf16 with M == 1 (the paper's V0-V7 shapes, appendix table "Matrix
 * shapes in our benchmark"), with the K rows split into num_splits ranges
 * that separate workgroups sum, so that shapes with few column strips
 * still occupy every CU.
 *
 *   A  device, bf16 [K]                       read only
 *   B  device, bf16 [K, N] row-major          read only
 *   C  device, [N]: fp32, or bf16 (rounded to nearest even once, from the
 *      fp32 sum) if c_bf16 != 0                written
 *   N % 64 == 0 and K % 8 == 0 (else TA_ERR_UNSUPPORTED)
 *   num_splits: 1..64 (else TA_ERR_INVALID_SHAPE); 1 runs gemm_bf16's
 *   matrix-vector kernel and ignores the workspace; for more, each range's
 *   fp32 partial sums go to `workspace` (device, 16-byte aligned, at least
 *   gemv_split_workspace_bytes(N, num_splits) bytes, owned by the caller, no
 *   overlap with A, B or C; TA_ERR_WORKSPACE if NULL or smaller) and a
 *   second kernel adds them in range order
 *   every pointer 16-byte aligned; C must not overlap A or B; stream as
 *   attn_fwd
 * Status codes as attn_fwd; validation before any HIP call.  The result
 * does not depend on timing; it differs from the unsplit kernel's in the
 * grouping of the fp32 additions only.
 */
ta_status gemv_bf16_split(const void *A, const void *B, void *C, int c_bf16, int N, int K,
                          int num_splits, void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes gemv_bf16_split needs: num_splits * N * 4 for
 * num_splits > 1, 0 for 1.  No HIP call. */
ta_status gemv_split_workspace_bytes(int N, int num_splits, size_t *bytes);

/* A split count for gemv_bf16_split.  A workgroup sums one strip of 256
 * columns (N % 256 == 0, else 64) over one K range, and two fit a CU; the
 * count chosen is the one whose workgroups (strips x splits, at most 512)
 * fill their last round of the 256 CUs most evenly, with at least 1024 rows
 * per range (fewer workgroups on a tie).  No HIP call. */
ta_status gemv_split_heuristic(int N, int K, int *num_splits);

/*
 * Mamba-2 state-space-duality (SSD) chunk functions: the paper's linear
 * attention workload ("chunk-scan and chunk-state functions from Mamba-2",
 * Section "Numerical Experiments", paragraph "Linear Attention Performance";
 * shapes in the appendix table "Linear Attention shapes in our benchmark").
 * For batch b, head h (group g = h / (nheads / ngroups)) and chunk c of
 * chunk_size positions, with a_l = sum_{l' <= l} dt_{l'} A_h the cumulative
 * log-decay inside the chunk (each call forms it from dt and A itself):
 *   ssd_chunk_state    S_c[p][n] = sum_l exp(a_last - a_l) dt_l x_l[p] Bm_l[n]
 *   ssd_state_passing  H_c = exp(a_last(c)) H_{c-1} + S_c, H_{-1} = 0; writes
 *                      the state each chunk enters with, H_{c-1}
 *   ssd_bmm_chunk      cb[l][s] = Cm_l . Bm_s (both positions in chunk c)
 *   ssd_chunk_scan     y_l[p] = exp(a_l) sum_n H_{c-1}[p][n] Cm_l[n]
 *                             + sum_{s <= l} cb[l][s] exp(a_l - a_s) dt_s x_s[p]
 *                             + D_h x_l[p]
 * Chained, they give the output of the recurrence h_t = exp(dt_t A) h_{t-1} +
 * dt_t x_t Bm_t^T, y_t = h_t Cm_t + D x_t (Mamba-2, "Transformers are SSMs").
 *
 * Layouts (contiguous, row-major; L = seqlen, nc = ceil(L / chunk_size)):
 *   x       device, bf16 [batch, L, nheads, headdim]
 *   Bm, Cm  device, bf16 [batch, L, ngroups, dstate]
 *   dt      device, fp32 [batch, L, nheads]           step sizes (> 0)
 *   A       device, fp32 [nheads]                     decay rates (<= 0)
 *   D       device, fp32 [nheads], or NULL for no skip term
 *   cb      device, fp32 [batch, nc, ngroups, chunk_size, chunk_size]
 *   states, prev_states
 *           device, fp32 [batch, nc, nheads, headdim, dstate]
 *   final_states device, fp32 [batch, nheads, headdim, dstate], or NULL
 *   out     device, fp32 [batch, L, nheads, headdim]
 * A last chunk shorter than chunk_size is handled as if padded with dt = 0
 * and zero x, Bm, Cm: padded positions add nothing (cb rows and columns of
 * padded positions are written as zero; out rows past L are not written).
 * headdim == 64, dstate == 128, chunk_size == 256 (else TA_ERR_UNSUPPORTED);
 * nheads % ngroups == 0 (else TA_ERR_INVALID_SHAPE).  bf16 and output
 * pointers 16-byte aligned, fp32 vectors 4-byte aligned (TA_ERR_MISALIGNED);
 * outputs must not overlap inputs (TA_ERR_ALIASING).  The decay- and
 * dt-weighted operand of each contraction (and, in the chunk scan, the fp32
 * entering state) is rounded to bf16 before the bf16 x bf16 -> fp32 MFMA.
 * Ownership, asynchrony and error behaviour as attn_fwd.
 */
ta_status ssd_chunk_state(const void *x, const void *Bm, const float *dt, const float *A,
                          float *states, int batch, int seqlen, int nheads, int ngroups,
                          int headdim, int dstate, int chunk_size, void *stream);

ta_status ssd_state_passing(const float *states, const float *dt, const float *A,
                            float *prev_states, float *final_states, int batch, int seqlen,
                            int nheads, int headdim, int dstate, int chunk_size, void *stream);

ta_status ssd_bmm_chunk(const void *Cm, const void *Bm, float *cb, int batch, int seqlen,
                        int ngroups, int dstate, int chunk_size, void *stream);

ta_status ssd_chunk_scan(const void *x, const void *Cm, const float *cb, const float *dt,
                         const float *A, const float *prev_states, const float *D, float *out,
                         int batch, int seqlen, int nheads, int ngroups, int headdim,
                         int dstate, int chunk_size, void *stream);

/*
 * ta_schedule — host-side tile schedule of attn_fwd, for tests and tools.
 * For the query tile `q_tile` (rows q_tile*BM .. q_tile*BM+BM-1, BM from
 * ta_tile_shape) it reports how many key tiles of BN keys the kernel visits
 * (n_kv_tiles; tiles past it are skipped because every key in them is
 * masked) and the first visited tile that needs per-element masking
 * (first_masked; == n_kv_tiles if none).  Pure integer logic, no HIP call.
 * Returns TA_ERR_INVALID_SHAPE for sizes < 1, q_tile out of range, or causal
 * with Sq > Sk; TA_ERR_UNSUPPORTED for D not 64/128; TA_ERR_NULL_POINTER.
 */
ta_status ta_schedule(int Sq, int Sk, int D, int causal, int q_tile,
                      int *n_kv_tiles, int *first_masked);

/* Query rows (BM) and keys (BN) per tile for head dim D; TA_ERR_UNSUPPORTED
 * for D not 64/128.  No HIP call. */
ta_status ta_tile_shape(int D, int *BM, int *BN);

/* Static text for a status code (never NULL). */
const char *ta_status_string(ta_status s);

/* Library version, major*10000 + minor*100 + patch. */
int ta_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TILEATTN_H */
