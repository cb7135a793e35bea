"""fp64 oracle for batched attention over a prefix forest (TEST INFRASTRUCTURE ONLY).

Parity status: every function here is pinned by the CPU tests in
``tests/test_oracle.py`` (brute force, closed forms, a library special case,
the shared == unshared identity and permutation invariances). The paper prints
no worked numeric example for attention, so no pin comes from a printed value.

Conventions (readings of points the paper leaves open):
  * scores are ``scale * <q, k>`` with ``scale`` supplied by the caller (the
    library uses the fp32-rounded 1/sqrt(d); the caller passes that value);
  * q head h reads kv head ``h // G`` with ``G = H_q // H_kv`` (contiguous
    groups);
  * a query with no visible key has output 0 and log-sum-exp -inf;
  * log-sum-exp is in natural log.

Inputs are numpy arrays; they are upcast to float64 exactly (bf16 and fp32
values are exactly representable in fp64).
"""

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def attend(q, k, v, scale, visible=None):
    """Scaled dot-product attention of n query rows over T keys, in fp64.

    Plain definition (textbook attention; the paper fixes only that sharing
    must not change it, §3 "Scope"):
        s[i, j]  = scale * sum_c q[i, c] * k[j, c]          for visible (i, j)
        m[i]     = max_j s[i, j]
        w[i, j]  = exp(s[i, j] - m[i]),  Z[i] = sum_j w[i, j]
        o[i, :]  = sum_j w[i, j] * v[j, :] / Z[i]
        lse[i]   = m[i] + ln Z[i]

    q: [n, d]; k, v: [T, d]; visible: optional [n, T] bool mask.
    Returns (o [n, d], lse [n]) as float64. Rows with no visible key get
    o = 0 and lse = -inf.
    """
    q = _f64(q)
    k = _f64(k)
    v = _f64(v)
    n, d = q.shape
    t = k.shape[0]
    o = np.zeros((n, v.shape[1] if v.ndim == 2 else d), dtype=np.float64)
    lse = np.full(n, -np.inf, dtype=np.float64)
    if n == 0 or t == 0:
        return o, lse
    s = float(scale) * (q @ k.T)
    if visible is not None:
        visible = np.asarray(visible, dtype=bool)
        s = np.where(visible, s, -np.inf)
        any_vis = visible.any(axis=1)
    else:
        any_vis = np.ones(n, dtype=bool)
    if not any_vis.any():
        return o, lse
    s = s[any_vis]
    m = s.max(axis=1, keepdims=True)
    w = np.exp(s - m)
    z = w.sum(axis=1)
    o[any_vis] = (w @ v) / z[:, None]
    lse[any_vis] = m[:, 0] + np.log(z)
    return o, lse


def attention_probs(q, k, scale, visible=None):
    """The softmax weights p[i, j] = exp(s[i, j] - lse[i]) of ``attend``.

    Exposed so tests can check that each row with a visible key sums to 1.
    """
    q = _f64(q)
    k = _f64(k)
    s = float(scale) * (q @ k.T)
    if visible is not None:
        s = np.where(np.asarray(visible, dtype=bool), s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    w = np.exp(s - m)
    z = w.sum(axis=1, keepdims=True)
    return np.divide(w, z, out=np.zeros_like(w), where=z > 0)


def _request_kv(seg_k, seg_v, path):
    """Concatenate the segments of one root-to-leaf path, prefix first.

    This is the unshared view of §2 ("Context reuse"): a request's context is
    its ancestors' context followed by its own tokens.
    """
    if len(path) == 0:
        return None, None
    ks = [_f64(seg_k[s]) for s in path]
    vs = [_f64(seg_v[s]) for s in path]
    return np.concatenate(ks, axis=0), np.concatenate(vs, axis=0)


def decode(q, seg_k, seg_v, req_paths, scale):
    """Decode attention: one query token per request, over all of its keys.

    q:        [R, H_q, d]
    seg_k[s]: [L_s, H_kv, d] logical keys of segment s (only the first L_s
              tokens; no page padding); seg_v likewise.
    req_paths: list of R lists of segment ids, root to leaf.
    Returns (o [R, H_q, d], lse [R, H_q]) float64.

    No key is masked in decode: the request's own newest token is part of its
    last segment (its K/V are written before attention runs).
    """
    q = _f64(q)
    r_count, h_q, d = q.shape
    o = np.zeros((r_count, h_q, d), dtype=np.float64)
    lse = np.full((r_count, h_q), -np.inf, dtype=np.float64)
    for r in range(r_count):
        k, v = _request_kv(seg_k, seg_v, req_paths[r])
        if k is None or k.shape[0] == 0:
            continue
        h_kv = k.shape[1]
        group = h_q // h_kv
        for g in range(h_kv):
            heads = slice(g * group, (g + 1) * group)
            oo, ll = attend(q[r, heads], k[:, g], v[:, g], scale)
            o[r, heads] = oo
            lse[r, heads] = ll
    return o, lse


def prefill(q, q_len, seg_k, seg_v, req_paths, scale):
    """Chunked prefill over a cached prefix (§4.1 prefix-caching discount).

    q:     [sum(q_len), H_q, d], request r's rows packed after those of r-1.
    q_len: [R] new tokens per request. The LAST segment of each path holds the
           K/V of exactly those new tokens (its length equals q_len[r]).
    Chunk query i (0-based) of request r sees every key of the earlier
    segments of its path and chunk keys j <= i.
    Returns (o [sum(q_len), H_q, d], lse [sum(q_len), H_q]).
    """
    q = _f64(q)
    total, h_q, d = q.shape
    o = np.zeros((total, h_q, d), dtype=np.float64)
    lse = np.full((total, h_q), -np.inf, dtype=np.float64)
    row0 = 0
    for r, path in enumerate(req_paths):
        n = int(q_len[r])
        if n == 0:
            continue
        k, v = _request_kv(seg_k, seg_v, path)
        t_total = k.shape[0]
        chunk = np.asarray(seg_k[path[-1]]).shape[0]
        if chunk != n:
            raise ValueError("last segment length must equal q_len")
        n_prefix = t_total - n
        i = np.arange(n)[:, None]
        j = np.arange(t_total)[None, :]
        visible = (j < n_prefix) | ((j - n_prefix) <= i)
        h_kv = k.shape[1]
        group = h_q // h_kv
        for h in range(h_q):
            g = h // group
            oo, ll = attend(q[row0:row0 + n, h], k[:, g], v[:, g], scale, visible)
            o[row0:row0 + n, h] = oo
            lse[row0:row0 + n, h] = ll
        row0 += n
    return o, lse


def merge_partials(os_, lses):
    """Combine attention results over disjoint key sets (exact in real numbers).

    For parts i with results (o_i, lse_i) over disjoint key sets, the result
    over their union is
        LSE = M + ln sum_i exp(lse_i - M),  M = max_i lse_i
        O   = sum_i exp(lse_i - LSE) * o_i
    Parts with lse = -inf contribute nothing; if all are -inf, O = 0 and
    LSE = -inf. Used by the tests to state the shared == unshared identity.
    os_: [P, n, d]; lses: [P, n].
    """
    os_ = _f64(os_)
    lses = _f64(lses)
    m = lses.max(axis=0)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    w = np.exp(lses - m_safe[None, :])
    z = w.sum(axis=0)
    lse = np.where(finite, m_safe + np.log(np.where(finite, z, 1.0)), -np.inf)
    coef = np.where(finite[None, :], np.exp(lses - np.where(finite, lse, 0.0)[None, :]), 0.0)
    o = (coef[:, :, None] * os_).sum(axis=0)
    return o, lse


def gather_tokens(seg_arrays, seq_list):
    """Expected output of the page gather: the logical tokens of each listed
    segment, concatenated in list order. seg_arrays[s] is [L_s, H_kv, d];
    returns [sum L, H_kv, d] with the input's dtype (a pure copy).
    """
    parts = [np.asarray(seg_arrays[s]) for s in seq_list]
    if not parts:
        return np.zeros((0,), dtype=np.float32)
    return np.concatenate(parts, axis=0)
