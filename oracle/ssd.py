"""float64 CPU oracle for the Mamba-2 SSD chunk functions.

TEST INFRASTRUCTURE, like the rest of this package: only the test suite, the
smoke check and the bench's CPU-baseline leg may import it.  It imports
nothing from the product; inputs come from the seeded generator as bfloat16
bit arrays (x, Bm, Cm) and float32 arrays (dt, A, D, cb, states).

What is computed.  The paper benchmarks the chunk-scan and chunk-state
functions of Mamba-2 as its linear-attention workload (Section "Numerical
Experiments", paragraph "Linear Attention Performance", and the appendix table
"Linear Attention shapes in our benchmark") without restating them; they are
the steps of Mamba-2's chunked state-space-duality (SSD) algorithm (Dao & Gu,
"Transformers are SSMs", 2024, Section 6).  For head h of batch b, with group
g = h // (H/G), position t, step dt_t > 0, decay rate A_h < 0 and the
recurrence

    h_t = exp(dt_t A_h) h_{t-1} + dt_t x_t Bm_t^T,    y_t = h_t Cm_t + D_h x_t

(h_t is P x N), the sequence is cut into chunks of Q positions and, with
a_l = sum_{l' <= l} dt_{l'} A_h the cumulative log-decay inside a chunk:

  1. chunk state   S_c = sum_{l in c} exp(a_last - a_l) dt_l x_l Bm_l^T
                   (the state a chunk would leave behind starting from zero)
  2. state passing H_c = exp(a_last of c) H_{c-1} + S_c, H_{-1} = 0; chunk c
                   enters with H_{c-1}
  3. chunk matrix  cb_c[l, s] = Cm_l . Bm_s
  4. chunk scan    y_l = exp(a_l) H_{c-1} Cm_l
                         + sum_{s <= l in c} cb[l, s] exp(a_l - a_s) dt_s x_s
                         + D_h x_l

Steps 1 and 4 are the two benchmarked functions; 2 and 3 complete the chain.
Everything below is that list of steps in float64, chunk by chunk, with
numpy's einsum forming the sums.  A ragged last chunk (L not a multiple of Q)
is padded with dt = 0 and zero x, Bm, Cm: a padded position adds nothing and
leaves the cumulative decay unchanged, so the last chunk's a_last is that of
its last real position.
"""
from __future__ import annotations

import numpy as np


class SsdOracleError(RuntimeError):
    pass


def _wide(bits):
    b = np.ascontiguousarray(bits)
    if b.dtype != np.uint16:
        raise TypeError("bf16 SSD inputs are bfloat16 bit arrays (numpy.uint16)")
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _chunked(a, Q, axis=1):
    """Pad axis `axis` (the sequence) with zeros to a multiple of Q and split
    it into (nc, Q)."""
    L = a.shape[axis]
    nc = -(-L // Q)
    pad = [(0, 0)] * a.ndim
    pad[axis] = (0, nc * Q - L)
    a = np.pad(a, pad)
    return a.reshape(a.shape[:axis] + (nc, Q) + a.shape[axis + 1:])


def dA_cumsum(dt, A, Q):
    """a[b, h, c, l] = sum_{l' <= l} dt[b, cQ + l', h] A[h]  (float64, [B, H, nc, Q])."""
    dt = np.asarray(dt, dtype=np.float64)
    A = np.asarray(A, dtype=np.float64)
    dtc = _chunked(dt, Q)                       # [B, nc, Q, H]
    return np.cumsum(dtc * A, axis=2).transpose(0, 3, 1, 2)


def _groups(H, G):
    if G < 1 or H % G:
        raise SsdOracleError(f"nheads {H} is not a multiple of ngroups {G}")
    return np.arange(H) // (H // G)


def chunk_state(x, Bm, dt, A, Q):
    """Step 1: S[b, c, h] (P x N) for every chunk, float64 [B, nc, H, P, N]."""
    X, Bw = _wide(x), _wide(Bm)
    Bsz, L, H, P = X.shape
    G, N = Bw.shape[2], Bw.shape[3]
    gmap = _groups(H, G)
    a = dA_cumsum(dt, A, Q)                                   # [B, H, nc, Q]
    dtc = _chunked(np.asarray(dt, dtype=np.float64), Q)       # [B, nc, Q, H]
    Xc = _chunked(X, Q)                                       # [B, nc, Q, H, P]
    Bc = _chunked(Bw, Q)[:, :, :, gmap, :]                    # [B, nc, Q, H, N]
    w = np.exp(a[:, :, :, -1:] - a) * dtc.transpose(0, 3, 1, 2)   # [B, H, nc, Q]
    return np.einsum("bhcl,bclhp,bclhn->bchpn", w, Xc, Bc)


def state_passing(states, dt, A, Q, initial=None):
    """Step 2: (entering states [B, nc, H, P, N], final state [B, H, P, N])."""
    S = np.asarray(states, dtype=np.float64)
    Bsz, nc, H, P, N = S.shape
    a = dA_cumsum(dt, A, Q)                                   # [B, H, nc, Q]
    if a.shape[2] != nc:
        raise SsdOracleError("states and dt disagree on the number of chunks")
    h = np.zeros((Bsz, H, P, N)) if initial is None else np.asarray(initial, dtype=np.float64)
    prev = np.empty_like(S)
    for c in range(nc):
        prev[:, c] = h
        h = np.exp(a[:, :, c, -1])[:, :, None, None] * h + S[:, c]
    return prev, h


def bmm_chunk(Cm, Bm, Q):
    """Step 3: cb[b, c, g, l, s] = Cm[cQ+l] . Bm[cQ+s], float64 [B, nc, G, Q, Q]."""
    Cc, Bc = _chunked(_wide(Cm), Q), _chunked(_wide(Bm), Q)   # [B, nc, Q, G, N]
    return np.einsum("bclgn,bcsgn->bcgls", Cc, Bc)


def chunk_scan(x, Cm, cb, dt, A, prev_states, D, Q):
    """Step 4: y float64 [B, L, H, P]."""
    X, Cw = _wide(x), _wide(Cm)
    Bsz, L, H, P = X.shape
    G = Cw.shape[2]
    gmap = _groups(H, G)
    a = dA_cumsum(dt, A, Q)                                   # [B, H, nc, Q]
    dtc = _chunked(np.asarray(dt, dtype=np.float64), Q).transpose(0, 3, 1, 2)   # [B, H, nc, Q]
    Xc = _chunked(X, Q)                                       # [B, nc, Q, H, P]
    Cc = _chunked(Cw, Q)[:, :, :, gmap, :]                    # [B, nc, Q, H, N]
    cbh = np.asarray(cb, dtype=np.float64)[:, :, gmap]        # [B, nc, H, Q, Q]
    Hin = np.asarray(prev_states, dtype=np.float64)           # [B, nc, H, P, N]
    # entering state, decayed to position l
    y = np.einsum("bchpn,bclhn->bclhp", Hin, Cc) * np.exp(a).transpose(0, 2, 3, 1)[..., None]
    # within the chunk: s <= l only
    Qn = a.shape[3]
    causal = np.tril(np.ones((Qn, Qn), dtype=bool))
    decay = np.where(causal, np.exp(np.where(causal, a[..., :, None] - a[..., None, :], 0.0)), 0.0)
    M = cbh * decay.transpose(0, 2, 1, 3, 4) * dtc.transpose(0, 2, 1, 3)[:, :, :, None, :]
    y = y + np.einsum("bchls,bcshp->bclhp", M, Xc)
    y = y + np.asarray(D, dtype=np.float64)[None, None, None, :, None] * Xc
    return y.reshape(Bsz, -1, H, P)[:, :L]


def chunk_scan_abs(x, Cm, cb, dt, A, prev_states, D, Q):
    """The same sums with every term replaced by its magnitude: the scale
    a rounding bound on the chunk-scan output is stated against."""
    absbits = lambda u: np.ascontiguousarray(u) & np.uint16(0x7FFF)
    return chunk_scan(absbits(x), absbits(Cm), np.abs(cb), dt, np.asarray(A), np.abs(prev_states),
                      np.abs(D), Q)


def chunk_state_abs(x, Bm, dt, A, Q):
    """|terms| version of chunk_state (the tolerance scale)."""
    absbits = lambda u: np.ascontiguousarray(u) & np.uint16(0x7FFF)
    return chunk_state(absbits(x), absbits(Bm), dt, A, Q)


def ssd_forward(x, dt, A, Bm, Cm, D, Q):
    """Steps 1-4 chained: y [B, L, H, P] and the final state [B, H, P, N]."""
    S = chunk_state(x, Bm, dt, A, Q)
    prev, final = state_passing(S, dt, A, Q)
    cb = bmm_chunk(Cm, Bm, Q)
    return chunk_scan(x, Cm, cb, dt, A, prev, D, Q), final
