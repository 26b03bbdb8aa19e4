"""Independent small-size references used to pin the oracle (tests only).

* ``brute_forward``: scalar Python loops with math.exp over the grouped
  problem written directly from Eq. (3) on each member sequence [P; R_i].
* ``packed_masked``: one masked attention over the packed sequence
  X_ours = [P; R_1; ...; R_G] (Eq. (2)) with the mask under which Eq. (4)
  equals Eq. (3) on every [P; R_i]: a prefix row sees the prefix keys up to
  itself, a response row sees the whole prefix and its own response up to
  itself. Gradients come from torch autograd (fp64, CPU), not from a
  hand-written backward.
"""
import math

import numpy as np


def brute_forward(prefix_lens, group_sizes, suffix_lens, t, scale):
    cu_p = np.concatenate([[0], np.cumsum(prefix_lens)])
    cu_s = np.concatenate([[0], np.cumsum(suffix_lens)])
    h_q, d = t["q_pre"].shape[1], t["q_pre"].shape[2]
    h_kv = t["k_pre"].shape[1]
    ratio = h_q // h_kv
    o_pre = np.zeros(t["q_pre"].shape)
    o_suf = np.zeros(t["q_suf"].shape)
    lse_pre = np.zeros((h_q, int(cu_p[-1])))
    lse_suf = np.zeros((h_q, int(cu_s[-1])))
    m = 0
    for g in range(len(prefix_lens)):
        p0, p1 = int(cu_p[g]), int(cu_p[g + 1])
        members = list(range(m, m + int(group_sizes[g])))
        m += int(group_sizes[g])

        def attend(qv, keys, vals):
            zs = [scale * sum(qv[c] * kk[c] for c in range(d)) for kk in keys]
            mx = max(zs)
            den = sum(math.exp(z - mx) for z in zs)
            lse = mx + math.log(den)
            out = [sum(math.exp(z - lse) * vv[c] for z, vv in zip(zs, vals)) for c in range(d)]
            return out, lse

        for h in range(h_q):
            kv = h // ratio
            for r in range(p0, p1):
                keys = [t["k_pre"][s, kv] for s in range(p0, r + 1)]
                vals = [t["v_pre"][s, kv] for s in range(p0, r + 1)]
                o, l_ = attend(t["q_pre"][r, h], keys, vals)
                o_pre[r, h] = o
                lse_pre[h, r] = l_
            for mm in members:
                s0, s1 = int(cu_s[mm]), int(cu_s[mm + 1])
                for r in range(s0, s1):
                    keys = [t["k_pre"][s, kv] for s in range(p0, p1)] + [t["k_suf"][s, kv] for s in range(s0, r + 1)]
                    vals = [t["v_pre"][s, kv] for s in range(p0, p1)] + [t["v_suf"][s, kv] for s in range(s0, r + 1)]
                    o, l_ = attend(t["q_suf"][r, h], keys, vals)
                    o_suf[r, h] = o
                    lse_suf[h, r] = l_
    return {"o_pre": o_pre, "o_suf": o_suf, "lse_pre": lse_pre, "lse_suf": lse_suf}


def packed_masked(torch, prefix_lens, group_sizes, suffix_lens, t, scale, grads=True):
    """Eq. (2) layout, one masked attention per group, gradients by autograd (fp64)."""
    cu_p = np.concatenate([[0], np.cumsum(prefix_lens)])
    cu_s = np.concatenate([[0], np.cumsum(suffix_lens)])
    h_q, d = t["q_pre"].shape[1], t["q_pre"].shape[2]
    h_kv = t["k_pre"].shape[1]
    ratio = h_q // h_kv
    leaves = {k: torch.tensor(np.asarray(v, dtype=np.float64), requires_grad=grads) for k, v in t.items()
              if not k.startswith("do")}
    outs = {"o_pre": torch.zeros(t["q_pre"].shape, dtype=torch.float64),
            "o_suf": torch.zeros(t["q_suf"].shape, dtype=torch.float64)}
    o_pre_parts, o_suf_parts = [], []
    m = 0
    loss = 0.0
    for g in range(len(prefix_lens)):
        p0, p1 = int(cu_p[g]), int(cu_p[g + 1])
        members = list(range(m, m + int(group_sizes[g])))
        m += int(group_sizes[g])
        s_lo = int(cu_s[members[0]]) if members else 0
        s_hi = int(cu_s[members[-1] + 1]) if members else 0
        x = {n: torch.cat([leaves[n + "_pre"][p0:p1], leaves[n + "_suf"][s_lo:s_hi]], 0) for n in ("q", "k", "v")}
        n_p, n = p1 - p0, (p1 - p0) + (s_hi - s_lo)
        # member id of each packed row: -1 for prefix rows
        owner = np.full(n, -1)
        pos = np.zeros(n, dtype=np.int64)
        pos[:n_p] = np.arange(n_p)
        for mm in members:
            a, b = int(cu_s[mm]) - s_lo + n_p, int(cu_s[mm + 1]) - s_lo + n_p
            owner[a:b] = mm
            pos[a:b] = np.arange(b - a)
        allowed = np.zeros((n, n), dtype=bool)
        for i in range(n):
            for j in range(n):
                if owner[j] == -1:  # prefix key
                    allowed[i, j] = owner[i] != -1 or j <= i
                else:
                    allowed[i, j] = owner[i] == owner[j] and pos[j] <= pos[i]
        mask = torch.tensor(np.where(allowed, 0.0, -np.inf))
        out = torch.zeros(n, h_q, d, dtype=torch.float64)
        outs_h = []
        for h in range(h_q):
            kv = h // ratio
            z = scale * x["q"][:, h, :] @ x["k"][:, kv, :].T + mask
            a = torch.softmax(z, dim=1)
            outs_h.append(a @ x["v"][:, kv, :])
        out = torch.stack(outs_h, dim=1)
        o_pre_parts.append(out[:n_p])
        o_suf_parts.append(out[n_p:])
    o_pre = torch.cat(o_pre_parts, 0)
    o_suf = torch.cat(o_suf_parts, 0)
    res = {"o_pre": o_pre.detach().numpy(), "o_suf": o_suf.detach().numpy()}
    if grads:
        loss = (o_pre * torch.tensor(np.asarray(t["do_pre"], np.float64))).sum() + \
               (o_suf * torch.tensor(np.asarray(t["do_suf"], np.float64))).sum()
        loss.backward()
        for n in ("q", "k", "v"):
            for side in ("pre", "suf"):
                gr = leaves[n + "_" + side].grad
                res["d%s_%s" % (n, side)] = (gr.numpy() if gr is not None
                                             else np.zeros(t[n + "_" + side].shape))
    return res
