"""GEMM-FLOP accounting of SequenceO1 Appendix G, restated.  TEST INFRASTRUCTURE.

Convention (Appendix G.1): FLOPs(U V) = 2 m r p for U in R^{m x r}, V in
R^{r x p}; SwiGLU with intermediate width w_f costs 6 T w w_f; lower-order
elementwise work (softmax exponentials, LayerNorm, ...) is not counted.

The sketching kernel's share of one SA layer is the affinity GEMM plus the
aggregation GEMM, 2 L_s L d + 2 L_s L d = 4 L_s L d (Appendix G.3); this is the
algorithmic FLOP count the benchmark reports per call (per head).
"""


def gemm(m, r, p):
    return 2.0 * m * r * p


def swiglu(T, w, wf):
    # Appendix G.1: two input projections and one output projection
    return gemm(T, w, wf) + gemm(T, w, wf) + gemm(T, wf, w)


def sa_layer(L, Ls, d):
    """Appendix G.3, per SA layer: 2 L d^2 + 14 L_s d^2 + 4 L_s L d."""
    key_proj = gemm(L, d, d)
    proto_proj = gemm(Ls, d, d)
    affinity = gemm(Ls, d, L)
    aggregation = gemm(Ls, L, d)
    ffn = swiglu(Ls, d, 2 * d)
    return key_proj + proto_proj + affinity + aggregation + ffn


def sa_kernel_term(L, Ls, d):
    """The part of one SA layer that the sketching kernel computes (affinity + aggregation)."""
    return gemm(Ls, d, L) + gemm(Ls, L, d)


def sa_total(L, n_sa, Ls, d):
    return n_sa * sa_layer(L, Ls, d)


def stca_layer_reordered(L, D, h):
    """Appendix G.2: single-query reordered attention 4 L D h + 6 D^2, plus W_O 2 D^2 and
    a one-token SwiGLU 12 D^2 -> 4 L D h + 20 D^2."""
    dh = D / h
    attn = h * (gemm(1, D, dh) + gemm(1, dh, D) + gemm(1, D, L) + gemm(1, L, D) + gemm(1, D, dh))
    return attn + gemm(1, D, D) + swiglu(1, D, 2 * D)


def stca_total(L, n_stca, D, h):
    """Per target: N (12 L D^2 + 4 L D h + 20 D^2) (history pre-FFN per layer included)."""
    return n_stca * (swiglu(L, D, 2 * D) + stca_layer_reordered(L, D, h))


def adapter(Ls, d, D):
    return gemm(Ls, d, D)


def seqo1_hit(Ls, d, D, n_stca, h):
    return adapter(Ls, d, D) + stca_total(Ls, n_stca, D, h)


def seqo1_expected(L, p_hit, n_sa, Ls, d, D, n_stca, h):
    return seqo1_hit(Ls, d, D, n_stca, h) + (1.0 - p_hit) * sa_total(L, n_sa, Ls, d)


def stca_mrlb(L, n_stca, D, h, R):
    """Only the per-layer history pre-FFNs are shared across the R targets."""
    shared = n_stca * swiglu(L, D, 2 * D)
    per_target = n_stca * stca_layer_reordered(L, D, h)
    return shared / R + per_target


def seqo1_mrlb_expected(L, R, p_hit, n_sa, Ls, d, D, n_stca, h):
    per_target = n_stca * stca_layer_reordered(Ls, D, h)
    shared = adapter(Ls, d, D) + n_stca * swiglu(Ls, D, 2 * D)
    return per_target + (shared + (1.0 - p_hit) * sa_total(L, n_sa, Ls, d)) / R
