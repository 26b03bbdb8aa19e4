"""Plain numpy oracle of grouped (shared-prefix) causal attention, forward and backward.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
bench's CPU baseline, never by the product path.

Definition followed (paper, Section 2.1):
* Eq. (1): member i of a group is the sequence x_i = [P; R_i] (no padding is
  needed here, every sequence is handled at its own length);
* Eq. (3): causal self-attention over x_i, O = softmax(scale * Q K^T + mask) V
  with the causal mask (query t sees keys 0..t, itself included);
* Eq. (4) and Lemma 1 (Appendix A.1, Eq. (9) and (13)): the grouped layer
  returns the prefix rows once and every suffix's rows; the gradient of the
  single shared prefix is the sum of the gradients that the G copies of the
  prefix receive in the repeated computation.

Readings taken where the paper is silent (all listed in the design notes):
* the log-sum-exp saved for the backward pass is the natural log of the
  softmax denominator, laid out [H_q, tokens];
* grouped-query attention maps query head h to key/value head
  h // (H_q / H_kv);
* the upstream gradient of a prefix row is split evenly over the G copies
  (dO_pre / G each): the grouped layer's prefix output is used once, so the
  copies must together carry exactly dO_pre; the 1/G that the proof writes in
  Eq. (9) is the GRPO loss weight, which lives in dO and is not applied again;
* a group with no members is its prefix alone, encoded once.

The softmax of a row is computed exactly over all the keys the row sees (no
running maximum, no tiling of the key axis). Rows are processed in chunks of
at most ``chunk`` rows purely to bound memory; a chunk never straddles the
prefix/suffix boundary, so every member computes its prefix rows with
identical operations.
"""
from __future__ import annotations

import numpy as np


def _kv_head(h: int, h_q: int, h_kv: int) -> int:
    if h_q % h_kv:
        raise ValueError("h_q must be a multiple of h_kv")
    return h // (h_q // h_kv)


def causal_attention(q, k, v, scale, do=None, split=None, chunk=1024, heads=None):
    """Causal self-attention over one sequence (Eq. (3)) and, if ``do`` is given, its gradient.

    q: [n, H_q, d]; k, v: [n, H_kv, d]; do: [n, H_q, d] (all one float dtype).
    ``split``: a row index that no row chunk may straddle (the prefix length).
    ``heads``: optional iterable of query heads to compute (others left zero).
    Returns dict with o [n, H_q, d], lse [H_q, n] and, with ``do``, dq, dk, dv.

    Forward, for each query head h (key/value head kv(h)) and row t:
      z_ts = scale * <q_t, k_s> for s <= t;  lse_t = ln sum_s exp(z_ts);
      a_ts = exp(z_ts - lse_t);              o_t = sum_s a_ts v_s.
    Backward (vector-Jacobian product of <do, o>):
      da_ts = <do_t, v_s>;  D_t = sum_s a_ts da_ts;  dz_ts = a_ts (da_ts - D_t);
      dq_t = scale * sum_s dz_ts k_s;  dk_s += scale * sum_t dz_ts q_t;
      dv_s += sum_t a_ts do_t   (dk, dv summed over the query heads sharing kv(h)).
    """
    n, h_q, d = q.shape
    h_kv = k.shape[1]
    dt = q.dtype
    out = {"o": np.zeros((n, h_q, d), dt), "lse": np.zeros((h_q, n), dt)}
    if do is not None:
        out["dq"] = np.zeros((n, h_q, d), dt)
        out["dk"] = np.zeros((n, h_kv, d), dt)
        out["dv"] = np.zeros((n, h_kv, d), dt)
    bounds = [0]
    for edge in ([split] if split not in (None, 0, n) else []) + [n]:
        while bounds[-1] < edge:
            bounds.append(min(edge, bounds[-1] + chunk))
    head_list = range(h_q) if heads is None else heads
    for h in head_list:
        kv = _kv_head(h, h_q, h_kv)
        for r0, r1 in zip(bounds[:-1], bounds[1:]):
            qs = q[r0:r1, h, :]
            ks = k[:r1, kv, :]
            vs = v[:r1, kv, :]
            z = scale * (qs @ ks.T)
            rows = np.arange(r0, r1)[:, None]
            cols = np.arange(r1)[None, :]
            z = np.where(cols <= rows, z, -np.inf)
            m = z.max(axis=1, keepdims=True)
            lse = m + np.log(np.exp(z - m).sum(axis=1, keepdims=True))
            a = np.exp(z - lse)
            out["o"][r0:r1, h, :] = a @ vs
            out["lse"][h, r0:r1] = lse[:, 0]
            if do is not None:
                dos = do[r0:r1, h, :]
                da = dos @ vs.T
                dd = (a * da).sum(axis=1, keepdims=True)
                dz = a * (da - dd)
                out["dq"][r0:r1, h, :] = scale * (dz @ ks)
                out["dk"][:r1, kv, :] += scale * (dz.T @ qs)
                out["dv"][:r1, kv, :] += a.T @ dos
    return out


def _group_members(group_sizes):
    start = np.concatenate([[0], np.cumsum(group_sizes)]).astype(np.int64)
    return [(int(start[g]), int(start[g + 1])) for g in range(len(group_sizes))]


def grouped_oracle(prefix_lens, group_sizes, suffix_lens, t, scale, grads=True, dtype=np.float64,
                   chunk=1024, heads=None, groups=None, check_members=True):
    """Grouped attention by the Repeated-Prefix Forward (Eq. (1), (3)) and Lemma 1.

    ``t`` maps q_pre, k_pre, v_pre, q_suf, k_suf, v_suf (and do_pre, do_suf when
    ``grads``) to float arrays in the packed varlen layout (``*_pre`` rows of
    group g at cu_prefix[g]:cu_prefix[g+1], ``*_suf`` rows of member m at
    cu_suffix[m]:cu_suffix[m+1], members of a group contiguous).

    For each group g with prefix P and members i = 1..G, the sequence
    [P; R_i] is encoded independently (Eq. (1)); the grouped results are
      o_pre, lse_pre   := the prefix rows of member 1 (all members agree, Lemma 1),
      o_suf, lse_suf   := the response rows of each member,
      d{q,k,v}_suf     := the response rows of each member's gradient,
      d{q,k,v}_pre     := sum over i = 1..G, in member order, of member i's prefix rows
    with member i receiving upstream gradient [do_pre / G; do_suf_i].

    ``heads`` restricts the query heads computed; ``groups`` restricts the
    groups (rows of other groups stay zero). Returns a dict of arrays plus
    ``prefix_member_spread``: the largest difference between any member's
    prefix outputs and member 1's (zero when the members agree bitwise).
    """
    g_members = _group_members(group_sizes)
    cu_p = np.concatenate([[0], np.cumsum(prefix_lens)]).astype(np.int64)
    cu_s = np.concatenate([[0], np.cumsum(suffix_lens)]).astype(np.int64)
    x = {name: np.asarray(a, dtype=dtype) for name, a in t.items()}
    h_q, d = x["q_pre"].shape[1], x["q_pre"].shape[2]
    h_kv = x["k_pre"].shape[1]
    tp, ts = int(cu_p[-1]), int(cu_s[-1])
    res = {"o_pre": np.zeros((tp, h_q, d), dtype), "o_suf": np.zeros((ts, h_q, d), dtype),
           "lse_pre": np.zeros((h_q, tp), dtype), "lse_suf": np.zeros((h_q, ts), dtype)}
    if grads:
        for side, n in (("pre", tp), ("suf", ts)):
            res["dq_" + side] = np.zeros((n, h_q, d), dtype)
            res["dk_" + side] = np.zeros((n, h_kv, d), dtype)
            res["dv_" + side] = np.zeros((n, h_kv, d), dtype)
    spread = 0.0
    group_list = range(len(prefix_lens)) if groups is None else groups
    for g in group_list:
        p0, p1 = int(cu_p[g]), int(cu_p[g + 1])
        m0, m1 = g_members[g]
        n_members = m1 - m0
        members = list(range(m0, m1)) if n_members else [None]
        share = 1.0 / n_members if n_members else 1.0
        for idx, m in enumerate(members):
            s0, s1 = (int(cu_s[m]), int(cu_s[m + 1])) if m is not None else (0, 0)

            def seq(name_pre, name_suf):
                return np.concatenate([x[name_pre][p0:p1], x[name_suf][s0:s1]], axis=0)

            q, k, v = seq("q_pre", "q_suf"), seq("k_pre", "k_suf"), seq("v_pre", "v_suf")
            do = None
            if grads:
                do = np.concatenate([x["do_pre"][p0:p1] * dtype(share), x["do_suf"][s0:s1]], axis=0)
            r = causal_attention(q, k, v, scale, do=do, split=p1 - p0, chunk=chunk, heads=heads)
            plen = p1 - p0
            if idx == 0:
                res["o_pre"][p0:p1] = r["o"][:plen]
                res["lse_pre"][:, p0:p1] = r["lse"][:, :plen]
            elif check_members and plen:
                spread = max(spread, float(np.abs(r["o"][:plen] - res["o_pre"][p0:p1]).max()),
                             float(np.abs(r["lse"][:, :plen] - res["lse_pre"][:, p0:p1]).max()))
            res["o_suf"][s0:s1] = r["o"][plen:]
            res["lse_suf"][:, s0:s1] = r["lse"][:, plen:]
            if grads:
                for name in ("dq", "dk", "dv"):
                    res[name + "_pre"][p0:p1] += r[name][:plen]
                    res[name + "_suf"][s0:s1] = r[name][plen:]
    res["prefix_member_spread"] = spread
    return res


def _member_of(cu_s, row):
    return int(np.searchsorted(cu_s, row, side="right") - 1)


def _group_of_member(group_sizes, m):
    start = np.concatenate([[0], np.cumsum(group_sizes)])
    return int(np.searchsorted(start, m, side="right") - 1)


def _group_of_prefix_row(cu_p, row):
    return int(np.searchsorted(cu_p, row, side="right") - 1)


def query_rows(prefix_lens, group_sizes, suffix_lens, t, scale, side, rows, heads, grads=True,
               dtype=np.float64, batch=256):
    """Outputs of selected query rows, each row from its own keys (Eq. (3) for one row).

    ``side`` is "pre" or "suf"; ``rows`` are packed row indices on that side;
    ``heads`` are query heads. A prefix row of group g at offset j sees prefix
    keys 0..j of its group; a suffix row at offset j of member i sees its
    group's whole prefix and response keys 0..j of member i ([P; R_i],
    Eq. (1)). For a prefix row the gradient is the sum over the G copies of
    the row, each carrying do_pre / G (Lemma 1); every copy sees the same keys
    and gives the same value, so the sum is G times one copy's.

    The requested rows are evaluated together where they read the same keys:
    the rows of one prefix (or one member's response) and the query heads of
    one key/value head form the rows of one matrix product over that
    sequence's keys, each row masked to the keys it sees; the softmax of every
    row is exact over its keys. ``batch`` bounds the rows of one product.

    Returns dict o [len(rows), len(heads), d], lse [len(heads), len(rows)]
    and, with ``grads``, dq like o.
    """
    cu_p = np.concatenate([[0], np.cumsum(prefix_lens)]).astype(np.int64)
    cu_s = np.concatenate([[0], np.cumsum(suffix_lens)]).astype(np.int64)
    h_q, d = t["q_pre"].shape[1], t["q_pre"].shape[2]
    h_kv = t["k_pre"].shape[1]
    rows = [int(r) for r in rows]
    heads = [int(h) for h in heads]
    nr, nh = len(rows), len(heads)
    o = np.zeros((nr, nh, d), dtype)
    lse = np.zeros((nh, nr), dtype)
    dq = np.zeros((nr, nh, d), dtype)
    f = lambda name, idx: np.asarray(t[name][idx], dtype)  # noqa: E731
    # owner of a row's key set: ("pre", group) or ("suf", member)
    owners = {}
    for a, row in enumerate(rows):
        key = ("pre", _group_of_prefix_row(cu_p, row)) if side == "pre" else ("suf", _member_of(cu_s, row))
        owners.setdefault(key, []).append(a)
    for (kind, idx), members in owners.items():
        last = max(rows[a] for a in members)
        if kind == "pre":
            g = idx
            p0 = int(cu_p[g])
            kk = f("k_pre", slice(p0, last + 1))
            vv = f("v_pre", slice(p0, last + 1))
            n_members = int(group_sizes[g])
            copies = max(1, n_members)
            share = 1.0 / n_members if n_members else 1.0
            limit = {a: rows[a] - p0 + 1 for a in members}  # keys seen by the row
            qn, don = "q_pre", "do_pre"
        else:
            m = idx
            g = _group_of_member(group_sizes, m)
            p0, p1 = int(cu_p[g]), int(cu_p[g + 1])
            s0 = int(cu_s[m])
            kk = np.concatenate([f("k_pre", slice(p0, p1)), f("k_suf", slice(s0, last + 1))], axis=0)
            vv = np.concatenate([f("v_pre", slice(p0, p1)), f("v_suf", slice(s0, last + 1))], axis=0)
            copies, share = 1, 1.0
            limit = {a: (p1 - p0) + rows[a] - s0 + 1 for a in members}
            qn, don = "q_suf", "do_suf"
        ridx = [rows[a] for a in members]
        qsel = f(qn, ridx)  # [rows, h_q, d]
        dosel = f(don, ridx) if grads else None
        for kv in sorted(set(_kv_head(h, h_q, h_kv) for h in heads)):
            hb = [b for b, h in enumerate(heads) if _kv_head(h, h_q, h_kv) == kv]
            # query vectors of this kv head: (row a, head b) pairs
            pairs = [(i, b) for i in range(len(members)) for b in hb]
            for c0 in range(0, len(pairs), batch):
                part = pairs[c0:c0 + batch]
                qm = np.stack([qsel[i, heads[b]] for i, b in part])
                lim = np.array([limit[members[i]] for i, _ in part])[:, None]
                z = scale * (qm @ kk[:, kv, :].T)
                z = np.where(np.arange(kk.shape[0])[None, :] < lim, z, -np.inf)
                mx = z.max(axis=1, keepdims=True)
                l_ = mx + np.log(np.exp(z - mx).sum(axis=1, keepdims=True))
                p = np.exp(z - l_)
                om = p @ vv[:, kv, :]
                if grads:
                    dom = np.stack([dosel[i, heads[b]] for i, b in part]) * dtype(share)
                    da = dom @ vv[:, kv, :].T
                    dz = p * (da - (p * da).sum(axis=1, keepdims=True))
                    dqm = scale * (dz @ kk[:, kv, :]) * dtype(copies)
                for j, (i, b) in enumerate(part):
                    a = members[i]
                    o[a, b] = om[j]
                    lse[b, a] = l_[j, 0]
                    if grads:
                        dq[a, b] = dqm[j]
    out = {"o": o, "lse": lse}
    if grads:
        out["dq"] = dq
    return out


def key_gradients(prefix_lens, group_sizes, suffix_lens, t, scale, group, kv_head, side, keys,
                  dtype=np.float64, chunk=1024, heads=None):
    """dK and dV of selected keys of one group and one key/value head.

    The gradient of key s is the sum over every query that sees s (Eq. (3)
    backward): dk_s = scale * sum_t dz_ts q_t and dv_s = sum_t a_ts do_t, over
    the query heads that share ``kv_head`` (or only ``heads`` if given). The
    queries of a prefix key are the group's prefix rows at or after it and
    every response row of every member; the queries of a response key are the
    rows of its own member at or after it.

    Each distinct query row is evaluated once, from its full key set. In the
    repeated computation a prefix row exists G times, every copy sees the same
    keys and carries do_pre / G, so the G copies together contribute exactly
    one evaluation with do_pre (the VJP is linear in dO; Lemma 1). This keeps
    the cost at the grouped size, which makes full-size workloads checkable.

    ``side`` is "pre" or "suf" and ``keys`` are packed row indices on that
    side (suffix keys must belong to ``group``). Returns dk, dv [len(keys), d].
    """
    cu_p = np.concatenate([[0], np.cumsum(prefix_lens)]).astype(np.int64)
    cu_s = np.concatenate([[0], np.cumsum(suffix_lens)]).astype(np.int64)
    g_members = _group_members(group_sizes)
    h_q, d = t["q_pre"].shape[1], t["q_pre"].shape[2]
    h_kv = t["k_pre"].shape[1]
    if heads is None:
        heads = [h for h in range(h_q) if _kv_head(h, h_q, h_kv) == kv_head]
    p0, p1 = int(cu_p[group]), int(cu_p[group + 1])
    plen = p1 - p0
    m0, m1 = g_members[group]
    keys = [int(s) for s in keys]
    dk = np.zeros((len(keys), d), dtype)
    dv = np.zeros((len(keys), d), dtype)
    kp = np.asarray(t["k_pre"][p0:p1, kv_head, :], dtype)
    vp = np.asarray(t["v_pre"][p0:p1, kv_head, :], dtype)

    def accumulate(q, do, k, v, first_row, n_rows, cols):
        # rows first_row .. first_row+n_rows-1 of a sequence whose key j is k[j]; row r sees keys 0..r.
        # Rows before the first selected key see none of them and are not evaluated.
        start = max(first_row, min(c for _, c in cols))
        for r0 in range(start, first_row + n_rows, chunk):
            r1 = min(first_row + n_rows, r0 + chunk)
            z = scale * (q[r0 - first_row:r1 - first_row] @ k[:r1].T)
            rows = np.arange(r0, r1)[:, None]
            z = np.where(np.arange(r1)[None, :] <= rows, z, -np.inf)
            mx = z.max(axis=1, keepdims=True)
            a = np.exp(z - (mx + np.log(np.exp(z - mx).sum(axis=1, keepdims=True))))
            dos = do[r0 - first_row:r1 - first_row]
            da = dos @ v[:r1].T
            dz = a * (da - (a * da).sum(axis=1, keepdims=True))
            qs = q[r0 - first_row:r1 - first_row]
            for j, c in cols:
                if c < r1:
                    dk[j] += scale * (dz[:, c] @ qs)
                    dv[j] += a[:, c] @ dos

    for h in heads:
        if side == "pre":
            cols = [(j, s - p0) for j, s in enumerate(keys)]
            qp = np.asarray(t["q_pre"][p0:p1, h, :], dtype)
            dop = np.asarray(t["do_pre"][p0:p1, h, :], dtype)
            accumulate(qp, dop, kp, vp, 0, plen, cols)
        for m in range(m0, m1):
            s0, s1 = int(cu_s[m]), int(cu_s[m + 1])
            if side == "pre":
                cols = [(j, s - p0) for j, s in enumerate(keys)]
            else:
                cols = [(j, plen + s - s0) for j, s in enumerate(keys) if s0 <= s < s1]
            if not cols or s1 == s0:
                continue
            k = np.concatenate([kp, np.asarray(t["k_suf"][s0:s1, kv_head, :], dtype)], 0)
            v = np.concatenate([vp, np.asarray(t["v_suf"][s0:s1, kv_head, :], dtype)], 0)
            qs = np.asarray(t["q_suf"][s0:s1, h, :], dtype)
            dos = np.asarray(t["do_suf"][s0:s1, h, :], dtype)
            accumulate(qs, dos, k, v, plen, s1 - s0, cols)
    return {"dk": dk, "dv": dv}
