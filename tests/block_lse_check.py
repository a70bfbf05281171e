"""Check of a stacked block's later-layer lse, split into its two error sources.

A later layer's logits use per-user prototypes P' = state W_Q W_K^T that the
device computes from its own state (rounded once to bf16 in bf16 mode).  So:
* the sketching step itself: the kernel's lse against the fp64 sketching
  oracle fed the device's own P' must meet the sketching step's own bound;
* the error of P' (the state's error from the earlier layers plus the
  rounding of P'): changing the prototypes by dP'_m moves lse_t by
  sum_m A_tm scale <X_t, dP'_m> for weights A on some point between the two
  (mean value theorem), so by at most scale |X_t| max_m |dP'_m|
  (Cauchy-Schwarz).  The oracle fed the device's P' and the block oracle must
  differ by no more than that, token by token.
"""
import numpy as np

import oracle
from oracle import block as oblock


def later_layer_lse(scale, X, P, params, offsets, Pp, lse, rlse, lse_tol, p_tol):
    """X [T,H,d], P [H,M,d], params = (Wq, Wk, ln, W1, W3, W2) with a leading
    layer axis, offsets [B+1] (host arrays of one batch or sub-batch); Pp[l] the
    device's P' of layer l for these users [B,H,M,d]; lse the device's and rlse
    the block oracle's [L,T,H] for these tokens."""
    off = np.asarray(offsets, np.int64)
    B = off.shape[0] - 1
    Wq, Wk = params[0], params[1]
    for l in range(1, lse.shape[0]):
        step = np.full(rlse[l].shape, np.nan)
        for b in range(B):
            t0, t1 = off[b], off[b + 1]
            if t1 > t0:
                step[t0:t1] = oracle.fwd(X[t0:t1], X[t0:t1], Pp[l][b], np.array([0, t1 - t0]), scale)[1]
        e_step = np.abs(lse[l] - step).max()
        print(f"layer {l}: lse of the sketching step on the device's P' {e_step:.3g}", flush=True)
        assert e_step <= lse_tol, ("lse of the sketching step", l, e_step)
        state = oblock.block_fwd(X, P, *[a[:l] for a in params], off, scale=scale)[0]
        Pr = np.einsum("bhmd,hde,hfe->bhmf", state, Wq[l].astype(np.float64), Wk[l].astype(np.float64))
        dmax = np.linalg.norm(Pp[l].astype(np.float64) - Pr, axis=3).max(axis=2)      # [B, H]
        user = np.repeat(np.arange(B), np.diff(off))
        bound = scale * np.linalg.norm(X.astype(np.float64), axis=2) * dmax[user]     # [T, H]
        gap = np.abs(step - rlse[l])
        print(f"layer {l}: lse moved by P' up to {gap.max():.3g} (bound {bound.max():.3g})", flush=True)
        assert np.all(gap <= bound * (1 + 1e-9) + 1e-12), ("lse moved by P' beyond its bound", l,
                                                            (gap - bound).max())
        rel = np.abs(Pp[l] - Pr).max(axis=(2, 3)) / np.abs(Pr).max(axis=(2, 3))
        assert np.all(rel <= p_tol), ("P'", l, rel.max())
