"""Brute-force scalar oracle (tiny shapes only).

TEST INFRASTRUCTURE ONLY.  The same method as ``oracle.wm`` written as plain
Python loops over scalars: no numpy reductions or matrix products, its own
Philox4x32-10 on Python integers and its own bfloat16 rounding through the
float32 bit pattern.  Agreement with the vectorised oracle on tiny shapes pins
the indexing, layouts and step order of both (a transposed operand, a wrong
gate block or a wrong stream index shows up as a disagreement).
"""

from __future__ import annotations

import math
import struct

_M0, _M1 = 0xD2511F53, 0xCD9E8D57
_W0, _W1 = 0x9E3779B9, 0xBB67AE85


def philox(c0, c1, c2, c3, k0, k1):
    """Philox4x32-10 (Salmon et al., SC'11) on Python integers."""
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _W0) & 0xFFFFFFFF
            k1 = (k1 + _W1) & 0xFFFFFFFF
        p0 = _M0 * c0
        p1 = _M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0) & 0xFFFFFFFF, p1 & 0xFFFFFFFF, \
            ((p0 >> 32) ^ c3 ^ k1) & 0xFFFFFFFF, p0 & 0xFFFFFFFF
    return c0, c1, c2, c3


def uniform(seed, traj, step, stream, index):
    """Uniform ``index`` of a stream: word index % 4 of block index // 4."""
    words = philox(index // 4, step & 0xFFFFFFFF, traj & 0xFFFFFFFF, stream,
                   seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    x = words[index % 4]
    return ((x >> 9) + 0.5) / 8388608.0


def bf16(x):
    """Nearest bfloat16 (ties to even) of float32(x), as a Python float."""
    bits = struct.unpack("<I", struct.pack("<f", x))[0]
    if math.isnan(x):
        return x
    bits = ((bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000) & 0xFFFFFFFF
    return struct.unpack("<f", struct.pack("<I", bits))[0]


def _q(x, dtype):
    return x if dtype == "fp32" else bf16(x)


def _sig(x):
    return 1.0 / (1.0 + math.exp(-x)) if x >= 0 else math.exp(x) / (1.0 + math.exp(x))


def _f32(x):
    return struct.unpack("<f", struct.pack("<f", x))[0]


def _argmax(scores, valid):
    best, bi = None, -1
    for i, s in enumerate(scores):
        if not valid[i]:
            continue
        s32 = _f32(s)
        if best is None or s32 > best:
            best, bi = s32, i
    return bi


def _mat(w, name, dtype):
    return [[_q(float(v), dtype) for v in row] for row in w[name]]


def _vec(w, name, dtype):
    return [_q(float(v), dtype) for v in w[name]]


def _step(w, Z, H, A, K, z, h, c, mask_row, seed, traj, s, tau, done_flag, dtype):
    Wg = _mat(w, "W_g", dtype)
    Wm = _mat(w, "W_m", dtype)
    Wc = _mat(w, "W_c", dtype)
    wr, wd = _vec(w, "w_r", dtype), _vec(w, "w_d", dtype)
    zq = [_q(v, dtype) for v in z]
    hq = [_q(v, dtype) for v in h]
    # controller (section 3.4) + masked Gumbel-max
    scores = []
    for a in range(A):
        acc = float(w["b_c"][a])
        for k in range(Z):
            acc += Wc[a][k] * zq[k]
        for k in range(H):
            acc += Wc[a][Z + k] * hq[k]
        scores.append(acc - math.log(-math.log(uniform(seed, traj, s, 0, a))))
    act = _argmax(scores, [m != 0 for m in mask_row])
    if act < 0:
        return None
    # gates + LSTM cell
    hn, cn = [0.0] * H, [0.0] * H
    for u in range(H):
        pre = []
        for gate in range(4):
            r = gate * H + u
            acc = float(w["b_g"][r]) + Wg[r][Z + act]
            for k in range(Z):
                acc += Wg[r][k] * zq[k]
            for k in range(H):
                acc += Wg[r][Z + A + k] * hq[k]
            pre.append(acc)
        cn[u] = _sig(pre[1]) * c[u] + _sig(pre[0]) * math.tanh(pre[2])
        hn[u] = _q(_sig(pre[3]) * math.tanh(cn[u]), dtype)
    # mixture head on h' (section 3.3.2)
    m = []
    for r in range(3 * Z * K):
        acc = float(w["b_m"][r])
        for k in range(H):
            acc += Wm[r][k] * hn[k]
        m.append(acc)
    zn = [0.0] * Z
    for j in range(Z):
        sc = []
        for k in range(K):
            sc.append(m[j * K + k] / tau
                      - math.log(-math.log(uniform(seed, traj, s, 1, j * K + k))))
        kk = _argmax(sc, [True] * K)
        p = j - (j % 2)
        r_ = math.sqrt(-2.0 * math.log(uniform(seed, traj, s, 2, p)))
        th = 2.0 * math.pi * uniform(seed, traj, s, 2, p + 1)
        eps = r_ * (math.cos(th) if j % 2 == 0 else math.sin(th))
        zn[j] = m[Z * K + j * K + kk] + math.exp(m[2 * Z * K + j * K + kk]) * eps
    rr = float(w["b_r"]) + sum(wr[k] * hn[k] for k in range(H))
    rd = float(w["b_d"]) + sum(wd[k] * hn[k] for k in range(H))
    d = False
    if done_flag:
        d = _f32(_sig(rd)) > _f32(uniform(seed, traj, s, 3, 0))
    return act, zn, hn, cn, rr, d


def rollout(w, dims, z0, mask, *, T, seed, tau=1.0, done_flag=True, dtype="fp32",
            traj0=0, step0=0, h0=None, c0=None, done0=None):
    """Scalar-loop dream rollout with the semantics of ``oracle.wm.rollout``."""
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    B = len(z0)
    out_z = [[[float(v) for v in z0[b]] for b in range(B)]]
    acts = [[-1] * B for _ in range(T)]
    rews = [[0.0] * B for _ in range(T)]
    dns = [[1] * B for _ in range(T)]
    zs = [[float(v) for v in z0[b]] for b in range(B)]
    hs = [[_q(float(h0[b][u]), dtype) if h0 is not None else 0.0 for u in range(H)]
          for b in range(B)]
    cs = [[float(c0[b][u]) if c0 is not None else 0.0 for u in range(H)] for b in range(B)]
    dn = [bool(done0[b]) if done0 is not None else False for b in range(B)]
    for t in range(T):
        for b in range(B):
            if dn[b]:
                continue
            r = _step(w, Z, H, A, K, zs[b], hs[b], cs[b], mask[b], seed, traj0 + b,
                      step0 + t, tau, done_flag, dtype)
            if r is None:
                dn[b] = True
                continue
            act, zn, hn, cn, rr, d = r
            acts[t][b], rews[t][b], dns[t][b] = act, rr, int(d)
            zs[b], hs[b], cs[b], dn[b] = zn, hn, cn, d
        out_z.append([list(zs[b]) for b in range(B)])
    return dict(z_out=out_z, actions=acts, rewards=rews, dones=dns, h_T=hs, c_T=cs,
                done_T=[int(x) for x in dn])


def controller_step(w, dims, z, h, mask, *, seed, step, traj0=0, dtype="fp32"):
    """Scalar-loop controller step: masked softmax probabilities and action."""
    Z, H, A = dims["Z"], dims["H"], dims["A"]
    Wc = _mat(w, "W_c", dtype)
    probs, actions = [], []
    for b in range(len(z)):
        zq = [_q(float(v), dtype) for v in z[b]]
        hq = [_q(float(v), dtype) for v in h[b]]
        logits = []
        for a in range(A):
            acc = float(w["b_c"][a])
            for k in range(Z):
                acc += Wc[a][k] * zq[k]
            for k in range(H):
                acc += Wc[a][Z + k] * hq[k]
            logits.append(acc)
        valid = [m != 0 for m in mask[b]]
        mx = max((logits[a] for a in range(A) if valid[a]), default=None)
        if mx is None:
            probs.append([0.0] * A)
        else:
            e = [math.exp(logits[a] - mx) if valid[a] else 0.0 for a in range(A)]
            s = sum(e)
            probs.append([v / s for v in e])
        sc = [logits[a] - math.log(-math.log(uniform(seed, traj0 + b, step, 0, a)))
              for a in range(A)]
        actions.append(_argmax(sc, valid))
    return dict(probs=probs, action=actions)


def nll(w, dims, z, actions, rewards, dones, *, lengths=None, dtype="fp32"):
    """Scalar-loop teacher-forced NLL with the semantics of ``oracle.wm.nll``."""
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    T, B = len(actions), len(actions[0])
    lengths = [T] * B if lengths is None else [min(max(int(x), 0), T) for x in lengths]
    Wg = _mat(w, "W_g", dtype)
    Wm = _mat(w, "W_m", dtype)
    wr, wd = _vec(w, "w_r", dtype), _vec(w, "w_d", dtype)
    ll = [[0.0] * B for _ in range(T)]
    se = [[0.0] * B for _ in range(T)]
    bce = [[0.0] * B for _ in range(T)]
    for b in range(B):
        h, c = [0.0] * H, [0.0] * H
        for t in range(T):
            zq = [_q(float(v), dtype) for v in z[t][b]]
            a = int(actions[t][b])
            hn, cn = [0.0] * H, [0.0] * H
            for u in range(H):
                pre = []
                for gate in range(4):
                    r = gate * H + u
                    acc = float(w["b_g"][r]) + (Wg[r][Z + a] if 0 <= a < A else 0.0)
                    for k in range(Z):
                        acc += Wg[r][k] * zq[k]
                    for k in range(H):
                        acc += Wg[r][Z + A + k] * h[k]
                    pre.append(acc)
                cn[u] = _sig(pre[1]) * c[u] + _sig(pre[0]) * math.tanh(pre[2])
                hn[u] = _q(_sig(pre[3]) * math.tanh(cn[u]), dtype)
            h, c = hn, cn
            if t >= lengths[b]:
                continue
            m = []
            for r in range(3 * Z * K):
                acc = float(w["b_m"][r])
                for k in range(H):
                    acc += Wm[r][k] * h[k]
                m.append(acc)
            tot = 0.0
            for j in range(Z):
                lp = [m[j * K + k] for k in range(K)]
                mx = max(lp)
                lse = mx + math.log(sum(math.exp(v - mx) for v in lp))
                terms = []
                for k in range(K):
                    mu, ls = m[Z * K + j * K + k], m[2 * Z * K + j * K + k]
                    x = float(z[t + 1][b][j])
                    terms.append(lp[k] - lse - 0.5 * ((x - mu) / math.exp(ls)) ** 2 - ls
                                 - 0.5 * math.log(2.0 * math.pi))
                mx = max(terms)
                tot += mx + math.log(sum(math.exp(v - mx) for v in terms))
            ll[t][b] = tot
            rr = float(w["b_r"]) + sum(wr[k] * h[k] for k in range(H))
            rd = float(w["b_d"]) + sum(wd[k] * h[k] for k in range(H))
            se[t][b] = (rr - float(rewards[t][b])) ** 2
            sp = max(rd, 0.0) + math.log1p(math.exp(-abs(rd)))
            bce[t][b] = sp - float(dones[t][b]) * rd
    N = sum(lengths)
    if N:
        means = [-sum(map(sum, ll)) / (N * Z), sum(map(sum, se)) / N, sum(map(sum, bce)) / N]
    else:
        means = [0.0, 0.0, 0.0]
    return dict(loglik=ll, reward_se=se, done_bce=bce, means=means)
