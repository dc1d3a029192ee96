"""Brute-force definitions used to pin the oracle (NumPy, fp64, tiny inputs only).

These take a different route from the oracle on purpose:
  * scores: the whole P x P causal attention matrix softmax(sigma Q K^T + mask)
    is built for every layer and head from queries at *every* position (the
    last one being the given q), and row P-1 is read out of it, as the paper
    describes reading the attention map returned by the prefill pass
    (Sec. 3.3, Eq. 6-8);
  * selection: the coverage distance of Eq. 10 is recomputed from scratch at
    every step from the full pairwise cosine matrix (no incremental update).
"""
import numpy as np
import scipy.special


def _f64(x, dtype):
    from paper_2607_27952_amd.workloads import as_f32
    return as_f32(x, dtype).astype(np.float64)


def scores(wl, rng=None, want_rows=False):
    rng = rng or np.random.default_rng(0)
    q = _f64(wl.q, wl.qk_dtype)
    k = _f64(wl.k, wl.qk_dtype)
    g = wl.Hq // wl.Hkv
    w = np.zeros(wl.N_total)
    rows = np.zeros((wl.G, wl.Hq, wl.T_total)) if want_rows else None
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        P = b - a
        v0, N = int(wl.vis_start[r]), wl.n(r)
        s = np.zeros(N)
        for l in range(wl.G):
            for h in range(wl.Hq):
                Kmat = k[l, a:b, h // g, :]                     # [P][Dh]
                Q = rng.standard_normal((P, wl.Dh))             # queries of earlier positions
                Q[P - 1] = q[l, r, h]
                logits = wl.scale * (Q @ Kmat.T)
                logits[np.triu_indices(P, 1)] = -np.inf         # causal mask
                A = scipy.special.softmax(logits, axis=1)
                row = A[P - 1]
                if want_rows:
                    rows[l, h, a:b] = row
                s += row[v0:v0 + N]
        w[int(wl.cu_vis[r]):int(wl.cu_vis[r + 1])] = s / s.sum()
    return (w, rows) if want_rows else w


def select(w32, X, K):
    """Greedy of Eq. 9-11 with delta recomputed from the full cosine matrix each step."""
    w = np.asarray(w32, dtype=np.float32).astype(np.float64)
    X = np.asarray(X, dtype=np.float64)
    n = np.linalg.norm(X, axis=1, keepdims=True)
    Xb = np.divide(X, n, out=np.zeros_like(X), where=n > 0)
    C = Xb @ Xb.T
    S = [int(np.argmax(w))]
    gains = [w[S[0]]]
    for _ in range(1, K):
        D = np.maximum(0.0, 1.0 - C[:, S])                    # [N][|S|]
        delta = D.min(axis=1)
        o = w * delta
        o[S] = -np.inf
        j = int(np.argmax(o))                                 # first maximum = lowest index
        S.append(j)
        gains.append(o[j])
    return np.array(S), np.array(gains)


def gonzalez(X, K):
    """Farthest-point (Gonzalez) k-center in cosine distance, starting at index 0."""
    X = np.asarray(X, dtype=np.float64)
    Xb = X / np.linalg.norm(X, axis=1, keepdims=True)
    dist = np.maximum(0.0, 1.0 - Xb @ Xb.T)
    S = [0]
    for _ in range(1, K):
        d = dist[:, S].min(axis=1)
        d[S] = -np.inf
        S.append(int(np.argmax(d)))
    return np.array(S)


def rows_scores(wl, cu_rows, row_pos, q_rows, rng=None, want_sums=False):
    """Table 4 sources by brute force: the full P x P causal attention matrix of
    every layer and head, with the given queries placed at their positions
    (random queries elsewhere); the listed rows are read out and summed, then
    normalised over the visual tokens (Eq. 7-8)."""
    rng = rng or np.random.default_rng(0)
    qr = _f64(q_rows, wl.qk_dtype)
    k = _f64(wl.k, wl.qk_dtype)
    g = wl.Hq // wl.Hkv
    w = np.zeros(wl.N_total)
    sums = np.zeros(wl.N_total)
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        P = b - a
        v0, N = int(wl.vis_start[r]), wl.n(r)
        rows = list(range(int(cu_rows[r]), int(cu_rows[r + 1])))
        s = np.zeros(N)
        for l in range(wl.G):
            for h in range(wl.Hq):
                Kmat = k[l, a:b, h // g, :]
                Q = rng.standard_normal((P, wl.Dh))
                for m in rows:
                    Q[int(row_pos[m])] = qr[l, m, h]
                logits = wl.scale * (Q @ Kmat.T)
                logits[np.triu_indices(P, 1)] = -np.inf
                A = scipy.special.softmax(logits, axis=1)
                for m in rows:
                    s += A[int(row_pos[m]), v0:v0 + N]
        sums[int(wl.cu_vis[r]):int(wl.cu_vis[r + 1])] = s
        w[int(wl.cu_vis[r]):int(wl.cu_vis[r + 1])] = s / s.sum()
    return (w, sums) if want_sums else w


def prefill(wl, q_all, v):
    """Causal prefill attention in matrix form: softmax(sigma Q K^T + causal mask) V
    for every layer, head and request (NumPy fp64)."""
    q = _f64(q_all, wl.qk_dtype)
    k = _f64(wl.k, wl.qk_dtype)
    vv = _f64(v, wl.qk_dtype)
    g = wl.Hq // wl.Hkv
    out = np.zeros(q.shape)
    for r in range(wl.R):
        a, b = int(wl.cu_seqlens[r]), int(wl.cu_seqlens[r + 1])
        P = b - a
        for l in range(wl.G):
            for h in range(wl.Hq):
                S = wl.scale * (q[l, a:b, h] @ k[l, a:b, h // g].T)
                S[np.triu_indices(P, 1)] = -np.inf
                out[l, a:b, h] = scipy.special.softmax(S, axis=1) @ vv[l, a:b, h // g]
    return out
