"""Shared test helpers: tolerances, comparisons and the oracle spec of a workload."""
import numpy as np

import oracle
from oracle.layer import Spec

# tolerance on activations: max|gpu - ref| / max|ref| per tensor
TOL = {"bf16": 2e-2, "f32": 1e-5}


def spec_of(w, mode=None):
    return Spec(w.n_heads, w.n_kv_heads, w.head_dim, w.block_size, w.top_k, mode or w.mode, w.dtype,
                w.rope_base, w.rms_eps)


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(got - ref))) / (den if den > 0 else 1.0)


def assert_close(got, ref, dtype, what="", tol=None):
    tol = TOL[dtype] if tol is None else tol
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    e = rel_err(got, ref)
    assert e <= tol, f"{what}: rel err {e:.3e} > {tol:.1e}"
    return e


def assert_close_with_infs(got, ref, dtype, what="", tol=None):
    """Infinite entries must coincide exactly; finite ones within tolerance."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    gi, ri = ~np.isfinite(got), ~np.isfinite(ref)
    assert np.array_equal(gi, ri), f"{what}: infinite entries differ ({int((gi != ri).sum())})"
    assert np.array_equal(got[gi], ref[ri]), f"{what}: signs of infinities differ"
    if np.any(~ri):
        return assert_close(got[~gi], ref[~ri], dtype, what, tol)
    return 0.0


def f64(a):
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# Selection parity.  Given the same Q/K bits, the selection is an exact
# integer function (exact fp64 scores, ties to the lower block), so the GPU's
# selection must equal the oracle's selector run on the GPU's own
# materialised Q/K (re-fed, bit-exact).  Against the oracle's own Q/K (which
# come from fp64 GEMMs instead of fp32-accumulated ones) a bf16 rounding can
# differ by one unit in the last place; a selected block may then differ
# only where the oracle's scores of the two blocks are closer than the
# change such roundings can cause.

def ulp(x, dtype):
    """Spacing of the activation dtype at |x| (its smallest spacing at 0)."""
    x = np.abs(np.asarray(x, dtype=np.float64))
    p, lo = (7, -133) if dtype == "bf16" else (23, -149)
    _, e = np.frexp(x)                       # x in [2^(e-1), 2^e)
    return np.where(x == 0, np.ldexp(1.0, lo), np.ldexp(1.0, np.maximum(e - 1 - p, lo)))


def _proj_bound(v, dv, W, dtype):
    """rho(W v) and the bound on its change when v moves by at most dv."""
    from oracle.selector import _project
    out = _project(v, W, dtype)
    dout = np.einsum("gkj,grj->grk", np.abs(W), dv) + ulp(out, dtype)
    return out, dout


def score_bounds(Q, K, B, G, dtype, ulps=1, w_gq=None, w_gk=None, kbar=None):
    """Exact scores r[Hkv, R, nf] of the oracle's selector and a bound on how
    far each can move when every element of Q[R, H, dh] and K[n, Hkv, dh]
    moves by at most `ulps` units in the last place (every rounding of the
    gate query and summary may then flip as well).  kbar [Hkv, nf, dh]: block
    summaries that both sides share exactly (K is then unused)."""
    from oracle.selector import block_summaries, gate_query, selector_scores
    Q = f64(Q)
    R, H, dh = Q.shape
    Hkv = H // G
    qh = gate_query(Q, G, dtype)                                     # [Hkv, R, dh]
    dq = ulps * ulp(Q, dtype).reshape(R, Hkv, G, dh).sum(axis=2).transpose(1, 0, 2) + ulp(qh, dtype)
    if w_gq is not None:
        qh, dq = _proj_bound(qh, dq, f64(w_gq), dtype)
    if kbar is not None:
        kb = f64(kbar)
        dk = np.zeros_like(kb)
    else:
        K = f64(K)
        kb = block_summaries(K, B, dtype)                            # [Hkv, nf, dh]
        nf = kb.shape[1]
        uk = ulp(K[:nf * B], dtype).reshape(nf, B, Hkv, dh).sum(axis=1).transpose(1, 0, 2)
        dk = ulps * uk / B + ulp(kb, dtype)
        if w_gk is not None:
            kb, dk = _proj_bound(kb, dk, f64(w_gk), dtype)
    r = selector_scores(qh, kb)
    bound = (np.einsum("grj,gmj->grm", dq, np.abs(kb)) + np.einsum("grj,gmj->grm", np.abs(qh), dk)
             + np.einsum("grj,gmj->grm", dq, dk))
    return r, bound


def assert_selection_near_ties(sel_gpu, sel_ref, r, bound, what=""):
    """sel_*[Hkv, R, K] of one sequence; r, bound [Hkv, R, nf].  Every block
    the GPU keeps instead of one the oracle keeps must be within the bound of
    it: r[a] - r[b] <= bound[a] + bound[b].  Returns the count of differing rows."""
    sel_gpu, sel_ref = np.asarray(sel_gpu), np.asarray(sel_ref)
    diff = np.nonzero(np.any(sel_gpu != sel_ref, axis=-1))
    for g, i in zip(*diff):
        a_set = set(int(m) for m in sel_ref[g, i] if m >= 0) - set(int(m) for m in sel_gpu[g, i] if m >= 0)
        b_set = set(int(m) for m in sel_gpu[g, i] if m >= 0) - set(int(m) for m in sel_ref[g, i] if m >= 0)
        assert len(a_set) == len(b_set), (what, g, i, sel_gpu[g, i], sel_ref[g, i])
        for a in a_set:
            for b in b_set:
                gap = r[g, i, a] - r[g, i, b]
                assert gap <= bound[g, i, a] + bound[g, i, b], \
                    (what, "row", int(i), "group", int(g), "blocks", a, b, "gap", gap, "bound",
                     bound[g, i, a] + bound[g, i, b])
    return len(diff[0])


def cache_keys(cache, bi, n):
    """K rows 0..n-1 of sequence bi from a paged GPU cache: [n, Hkv, dh] (float64)."""
    import torch
    ps = cache.page_size
    t = np.arange(n)
    pages = cache.block_table[bi].cpu().numpy()[t // ps]
    kp = cache.k_pages[torch.from_numpy(pages.astype(np.int64)).to(cache.k_pages.device), :,
                       torch.from_numpy((t % ps).astype(np.int64)).to(cache.k_pages.device)]
    return f64(kp.float().cpu().numpy())


def check_decode_selection(sel_gpu, q_gpu, cache, pos, spec, ocache=None, bsel=None, q_ref=None,
                           w_gq=None, w_gk=None, summaries_from_keys=True):
    """Selection parity of a decode step.  sel_gpu [b, Hkv, K] (host), q_gpu
    [b, H, dh] the step's query-head tap (device), cache the GPU's paged
    cache after the step, pos an int or [b] positions.
    * Re-fed: the oracle's decode selection on the GPU's own query heads and
      cached summaries equals the GPU's, bit-exact (every sequence).
    * Summaries: the GPU's cached summaries of the complete blocks equal the
      oracle's summaries of the GPU's cached keys, bit-exact (no projection).
    * Raw (when the oracle's cache `ocache` and its query heads q_ref are given,
      for the sequences `bsel`): rows that differ from the oracle's own
      selection do so only at near-ties within one ulp of Q/K.
    summaries_from_keys=False: the caches' summaries were written directly
    (not pooled from the cached keys) and are the same on both sides."""
    import oracle
    from oracle.selector import block_summaries
    b = sel_gpu.shape[0]
    pos = np.full(b, pos) if np.ndim(pos) == 0 else np.asarray(pos)
    qg = f64(q_gpu.float().cpu().numpy())
    kbar = f64(cache.k_summary.float().cpu().numpy())
    ref, _ = oracle.decode_select(qg, pos, kbar, spec, w_gq=w_gq)
    np.testing.assert_array_equal(sel_gpu, ref)
    B = spec.block_size
    if w_gk is None and summaries_from_keys:
        for bi in range(b):
            nb = int(pos[bi] + 1) // B
            if nb:
                np.testing.assert_array_equal(kbar[bi, :, :nb], block_summaries(cache_keys(cache, bi, nb * B), B,
                                                                                spec.dtype))
    nd = 0
    if ocache is not None:
        bsel = list(range(b)) if bsel is None else list(bsel)
        selo, _ = oracle.decode_select(q_ref, pos[bsel], ocache.kbar, spec, w_gq=w_gq)
        for j, bi in enumerate(bsel):
            ct = int(pos[bi]) // B
            if ct == 0:
                continue
            r, bd = score_bounds(q_ref[j][None], ocache.K[j, :ct * B], B, spec.group, spec.dtype,
                                 w_gq=w_gq, w_gk=w_gk,
                                 kbar=None if summaries_from_keys else ocache.kbar[j][:, :ct])
            nd += assert_selection_near_ties(sel_gpu[bi][:, None], selo[j][:, None], r, bd, f"decode t={pos[bi]}")
    return nd
