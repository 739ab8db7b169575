"""Planted mistakes in the oracle must each trip at least one pin.

Every mutation replaces one oracle function with a plausibly wrong variant
(a dropped or wrong term, an off-by-one, a transposed operand, a flipped
sign); the pin battery then has to fail.  Runs on the CPU only.
"""
import numpy as np
import pytest

from oracle import dfa_oracle as O
from tests import oracle_pins as pins

# cheap pins first: a mutation stops at the first pin that catches it
ORDER = ["P4", "P3", "P6", "P7", "P5", "P8", "P9", "P10", "P12", "P13", "P14", "P15", "P2", "P1", "P16",
         "P11"]


def _probs_factory(scale_fn=None, transpose=False, axis=-1):
    def probs(q, k, w=None, rows=None):
        q = np.asarray(q, dtype=np.float64)
        k = np.asarray(k, dtype=np.float64)
        L, d = k.shape
        if rows is None:
            rows = np.arange(q.shape[0])
        S = (q @ k.T) * (scale_fn(d) if scale_fn else 1.0 / np.sqrt(d))
        if transpose:
            S = S.T[:q.shape[0]] if S.shape[0] == S.shape[1] else S
        mask = None if w is None else O.band_mask(rows, L, w)
        if mask is not None:
            S = np.where(mask, S, -np.inf)
        E = np.exp(S - np.max(S, axis=-1, keepdims=True))
        return E / np.sum(E, axis=axis, keepdims=True)
    return probs


def _band_strict(rows, L, w):
    j = np.arange(L)
    return np.abs(np.asarray(rows)[:, None] - j[None, :]) < w


def _band_wrap(rows, L, w):
    j = np.arange(L)
    dist = np.abs(np.asarray(rows)[:, None] - j[None, :])
    return np.minimum(dist, L - dist) <= w


def _band_shifted(rows, L, w):
    # constant-width window slid inward at the sequence ends
    rows = np.asarray(rows)
    lo = np.clip(rows - w, 0, max(0, L - 1 - 2 * w))
    j = np.arange(L)
    return (j[None, :] >= lo[:, None]) & (j[None, :] <= lo[:, None] + 2 * w)


def _n_band_no_trunc(L, w):
    return L * (2 * w + 1)


def _refresh_sign(Q, K, V, w):
    Of = O.attn_full(Q, K, V)
    return Of, O.attn_window(Q, K, V, w) - Of


def _reuse_on_full(Q, K, V, R, w):
    return O.attn_full(Q, K, V) + R


def _asc_uncond_source(Q, K, V):
    half = np.shape(Q)[0] // 2
    Ou = O.attn_full(np.asarray(Q)[half:], np.asarray(K)[half:], np.asarray(V)[half:])
    return np.concatenate([Ou, Ou], axis=0)


def _wars_asc_uncond_source(Q, K, V, w):
    half = np.shape(Q)[0] // 2
    Ou, Ru = O.wars_refresh(np.asarray(Q)[half:], np.asarray(K)[half:], np.asarray(V)[half:], w)
    return np.concatenate([Ou, Ou], axis=0), Ru


def _wars_asc_reuse_no_residual(Q, K, V, R_cond, w):
    half = np.shape(Q)[0] // 2
    Oc = O.attn_window(np.asarray(Q)[:half], np.asarray(K)[:half], np.asarray(V)[:half], w)
    return np.concatenate([Oc, Oc], axis=0)


def _residual_wrong_half(code, cache, B):
    if cache.R is None:
        raise ValueError("reuse before any refresh")
    return cache.R if code == O.WARS_REUSE else cache.R[-(B // 2):]


def _residual_unchecked(code, cache, B):
    if cache.R is None:
        raise ValueError("reuse before any refresh")
    return cache.R if code == O.WARS_REUSE else cache.R[: B // 2]


def _qkv_split_heads_first(X, Wqkv, bqkv, H):
    X = np.asarray(X, dtype=np.float64)
    B, L, C = X.shape
    Y = (X @ np.asarray(Wqkv).T + bqkv).reshape(B, L, H, 3, C // H)   # (h, which) swapped
    return tuple(np.ascontiguousarray(Y[:, :, :, i].transpose(0, 2, 1, 3)) for i in range(3))


def _out_merge_dims_first(O_, Wo, bo):
    O_ = np.asarray(O_, dtype=np.float64)
    B, H, L, d = O_.shape
    return O_.transpose(0, 2, 3, 1).reshape(B, L, H * d) @ np.asarray(Wo).T + bo   # (dim, head) order


def _out_weight_transposed(O_, Wo, bo):
    O_ = np.asarray(O_, dtype=np.float64)
    B, H, L, d = O_.shape
    return O_.transpose(0, 2, 1, 3).reshape(B, L, H * d) @ np.asarray(Wo) + bo


def _qkv_no_bias(X, Wqkv, bqkv, H):
    return _orig_qkv(X, Wqkv, None, H)


_orig_qkv = O.qkv_proj
_orig_module_step = O.module_step


def _module_asc_projects_whole_batch(code, X, wts, cache, w):
    if code == O.ASC_REUSE:
        Y = O.out_proj(O.attn_full(*O.qkv_proj(X, wts.Wqkv, wts.bqkv, wts.H)), wts.Wo, wts.bo)
        half = np.shape(X)[0] // 2
        Y = np.concatenate([Y[half:], Y[half:]], axis=0)
        cache.Y_cache = Y
        return Y
    return _orig_module_step(code, X, wts, cache, w)


def _mrae_no_abs(Oa, Ob, eps=O.MRAE_EPS):
    a = np.asarray(Oa, dtype=np.float64).ravel()
    b = np.asarray(Ob, dtype=np.float64).ravel()
    return float(np.mean(np.clip((a - b) / (np.maximum(a, b) + eps), 0.0, 10.0)))


def _mrae_min_norm(Oa, Ob, eps=O.MRAE_EPS):
    a = np.asarray(Oa, dtype=np.float64).ravel()
    b = np.asarray(Ob, dtype=np.float64).ravel()
    return float(np.mean(np.clip(np.abs(a - b) / (np.minimum(np.abs(a), np.abs(b)) + eps), 0.0, 10.0)))


def _order_reversed(L, C, w):
    return tuple(reversed(_orig_order(L, C, w)))


_orig_order = O.strategy_order
_orig_search = O.plan_search


def _search_zero_based_threshold(X_steps, layers, delta, w, store=None):
    # (i / |M|) delta with a 0-based layer index: layer 0 can never be compressed
    import copy
    n_layers = len(layers)
    B, L, C = np.shape(X_steps[0])
    order = O.strategy_order(L, C, w)
    caches = [O.ModuleCache() for _ in range(n_layers)]
    plan = np.full((len(X_steps), n_layers), -1, dtype=np.int32)
    loss = np.full(plan.shape, np.nan)
    for t, X in enumerate(X_steps):
        X = np.asarray(X, dtype=np.float64)
        O_ref = O.surrogate_forward(X, layers, [O.FULL] * n_layers, [O.ModuleCache() for _ in layers], w)
        for i in range(n_layers):
            chosen = O.WARS_REFRESH
            for m in order:
                if not O._applicable(m, caches[i], B):
                    continue
                trial = copy.deepcopy(caches[i])
                Xi = X + O.module_step(m, X, layers[i], trial, w)
                O2 = O.surrogate_forward(Xi, layers, [O.FULL] * n_layers, [O.ModuleCache() for _ in layers], w,
                                         first=i + 1)
                if O.mrae(O_ref, O2) < i / n_layers * delta:
                    chosen = m
                    break
            plan[t, i] = chosen
            X = X + O.module_step(chosen, X, layers[i], caches[i], w)
    return plan, loss


def _search_stale_reference(X_steps, layers, delta, w, store=None):
    # the uncompressed output of step 0 serves as the reference of every step
    return _search_with_reference(X_steps, layers, delta, w, stale=True)


def _search_commit_full(X_steps, layers, delta, w, store=None):
    # uncompressed layers committed as FULL: no residual is ever refreshed
    return _search_with_reference(X_steps, layers, delta, w, commit_full=True)


def _search_with_reference(X_steps, layers, delta, w, stale=False, commit_full=False):
    import copy
    n_layers = len(layers)
    B, L, C = np.shape(X_steps[0])
    order = O.strategy_order(L, C, w)
    caches = [O.ModuleCache() for _ in range(n_layers)]
    plan = np.full((len(X_steps), n_layers), -1, dtype=np.int32)
    loss = np.full(plan.shape, np.nan)
    O_first = None
    for t, X in enumerate(X_steps):
        X = np.asarray(X, dtype=np.float64)
        O_ref = O.surrogate_forward(X, layers, [O.FULL] * n_layers, [O.ModuleCache() for _ in layers], w)
        if stale:
            O_first = O_ref if O_first is None else O_first
            O_ref = O_first
        for i in range(n_layers):
            chosen = O.FULL if commit_full else O.WARS_REFRESH
            for m in order:
                if not O._applicable(m, caches[i], B):
                    continue
                trial = copy.deepcopy(caches[i])
                Xi = X + O.module_step(m, X, layers[i], trial, w)
                O2 = O.surrogate_forward(Xi, layers, [O.FULL] * n_layers, [O.ModuleCache() for _ in layers], w,
                                         first=i + 1)
                if O.mrae(O_ref, O2) < (i + 1) / n_layers * delta:
                    chosen = m
                    break
            plan[t, i] = chosen
            X = X + O.module_step(chosen, X, layers[i], caches[i], w)
    return plan, loss


_orig_plan_step = O.plan_step


def _plan_step_full_clears_R(code, Q, K, V, cache, w):
    out = _orig_plan_step(code, Q, K, V, cache, w)
    if code == O.FULL:
        cache.R = None if cache.R is None else np.zeros_like(cache.R)
    return out


_orig_plan_make = O.plan_make


class _SplitMixTypo(O.SplitMix64):
    def next(self):
        self.state = (self.state + 0x9E3779B97F4A7C15) & O._MASK64
        z = self.state
        z = ((z ^ (z >> 31)) * 0xBF58476D1CE4E5B9) & O._MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & O._MASK64
        return z ^ (z >> 31)


def _plan_age_off_by_one(seed, n_layers, n_steps, refresh_every, B):
    rng = O.SplitMix64(seed)
    code = np.full((n_steps, n_layers), -1, dtype=np.int32)
    r_src = np.full_like(code, -1)
    o_src = np.full_like(code, -1)
    last, cache = [-1] * n_layers, [-1] * n_layers
    for t in range(n_steps):
        for l in range(n_layers):
            c = ((rng.next() >> 32) * 5) >> 32
            if c == O.AST_REUSE and cache[l] < 0:
                c = O.FULL
            if refresh_every > 0 and c in (1, 2):
                c = 1 if (last[l] < 0 or t - last[l] > refresh_every) else 2  # '>' for '>='
            if refresh_every == 0 and c == 2 and last[l] < 0:
                c = 1
            code[t, l] = c
            if c == 2:
                r_src[t, l] = last[l]
            if c == 3:
                o_src[t, l] = cache[l]
            else:
                o_src[t, l] = t
                cache[l] = t
            if c == 1:
                last[l] = t
    return code, r_src, o_src


def _plan_ast_at_start(seed, n_layers, n_steps, refresh_every, B):
    code, r_src, o_src = _orig_plan_make(seed, n_layers, n_steps, refresh_every, B)
    code = code.copy()
    code[0, 0] = O.AST_REUSE
    return code, r_src, o_src


def _rows_block_local(Q, K, V, rows, w=None):
    # the band built from indices within the row block instead of token indices
    Q, K, V = (np.asarray(x, dtype=np.float64) for x in (Q, K, V))
    rows = np.asarray(rows, dtype=np.int64)
    B, H, L, d = Q.shape
    out = np.empty((B, H, len(rows), d))
    for b in range(B):
        for h in range(H):
            for r0 in range(0, len(rows), O._ROW_BLOCK):
                rr = rows[r0:r0 + O._ROW_BLOCK]
                P = O.attention_probs(Q[b, h, rr], K[b, h], w, np.arange(len(rr)))
                out[b, h, r0:r0 + len(rr)] = P @ V[b, h]
    return out


_plan_step_rows = O.plan_step_rows


def _rows_reuse_on_full(code, Q, K, V, rows, cache, w):
    # the sampled reuse step evaluated on full attention instead of the window
    if code == O.WARS_REUSE:
        Ofull = O.attention_rows(Q, K, V, rows, None) + O._residual_for(code, cache, np.shape(Q)[0])
        cache.O_cache = Ofull
        return Ofull
    return _plan_step_rows(code, Q, K, V, rows, cache, w)


MUTATIONS = {
    "scale_1_over_d": ("attention_probs", _probs_factory(scale_fn=lambda d: 1.0 / d)),
    "scale_missing": ("attention_probs", _probs_factory(scale_fn=lambda d: 1.0)),
    "scores_transposed": ("attention_probs", _probs_factory(transpose=True)),
    "softmax_wrong_axis": ("attention_probs", _probs_factory(axis=0)),
    "band_strict": ("band_mask", _band_strict),
    "band_wraps": ("band_mask", _band_wrap),
    "band_shifted_at_edges": ("band_mask", _band_shifted),
    "band_count_untruncated": ("n_band", _n_band_no_trunc),
    "residual_sign": ("wars_refresh", _refresh_sign),
    "reuse_adds_to_full": ("wars_reuse", _reuse_on_full),
    "asc_wrong_half": ("asc_reuse", _asc_uncond_source),
    "wars_asc_wrong_half": ("wars_asc_refresh", _wars_asc_uncond_source),
    "wars_asc_reuse_drops_residual": ("wars_asc_reuse", _wars_asc_reuse_no_residual),
    "wars_asc_reads_uncond_residual": ("_residual_for", _residual_wrong_half),
    "half_residual_feeds_full_reuse": ("_residual_for", _residual_unchecked),
    "qkv_split_heads_first": ("qkv_proj", _qkv_split_heads_first),
    "qkv_bias_dropped": ("qkv_proj", _qkv_no_bias),
    "out_merge_dims_first": ("out_proj", _out_merge_dims_first),
    "out_weight_transposed": ("out_proj", _out_weight_transposed),
    "module_asc_uses_uncond_half": ("module_step", _module_asc_projects_whole_batch),
    "mrae_without_abs": ("mrae", _mrae_no_abs),
    "mrae_min_normaliser": ("mrae", _mrae_min_norm),
    "search_order_reversed": ("strategy_order", _order_reversed),
    "search_zero_based_threshold": ("plan_search", _search_zero_based_threshold),
    "search_stale_reference": ("plan_search", _search_stale_reference),
    "search_commit_full": ("plan_search", _search_commit_full),
    "full_clears_residual": ("plan_step", _plan_step_full_clears_R),
    "splitmix_shift_typo": ("SplitMix64", _SplitMixTypo),
    "refresh_age_off_by_one": ("plan_make", _plan_age_off_by_one),
    "ast_at_first_step": ("plan_make", _plan_ast_at_start),
    "rows_band_block_local": ("attention_rows", _rows_block_local),
    "rows_reuse_on_full": ("plan_step_rows", _rows_reuse_on_full),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, repl = MUTATIONS[name]
    monkeypatch.setattr(O, attr, repl)
    caught = None
    for pin in ORDER:
        try:
            with np.errstate(all="ignore"):
                pins.ALL_PINS[pin]()
        except (AssertionError, ValueError, FloatingPointError, IndexError):
            caught = pin
            break
    assert caught is not None, f"planted mistake {name!r} passed every pin"
