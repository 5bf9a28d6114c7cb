"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each ``pin_*`` takes an ``oracle.Oracle`` handle and raises AssertionError when
the oracle disagrees with an independent fact: a closed form of a special
case, brute force on tiny inputs, a library routine the special case reduces
to, or an invariant of the method.  None retypes the oracle's own formula.
The same pins run against deliberately broken copies of the oracle
(``test_oracle_mutants.py``), each of which must fail at least one pin.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import torch

import synth

SCALE = float(np.float32(1.0 / math.sqrt(128.0)))


# --- bf16 helpers (host side, used only to build inputs) ----------------------
def f2bf(x) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest even (finite inputs)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def bf2f(u) -> np.ndarray:
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def rand_bf(rng, shape, scale=1.0):
    return f2bf(rng.standard_normal(shape) * scale)


# --- bf16 decode --------------------------------------------------------------
def pin_bf16_decode(orc):
    cases = {0x3F80: 1.0, 0xC000: -2.0, 0x4049: 3.140625, 0x0001: 2.0 ** -133,
             0x8000: -0.0, 0x7F80: math.inf, 0x3E00: 0.125, 0x4500: 2048.0}
    for bits, val in cases.items():
        got = orc.bf16_to_f64(bits)
        assert got == val, (hex(bits), got, val)


# --- scores -------------------------------------------------------------------
def pin_scores_onehot(orc):
    """Query heads that are one-hot on distinct channels: each head's logit is
    scale * value * K[j, c_g], and the group's score is the largest of them."""
    rng = np.random.default_rng(1)
    G, d, n = 4, 128, 61
    K = rand_bf(rng, (n, d))
    chans, vals = [5, 77, 3, 127], [1.0, -2.0, 0.5, 3.0]
    q = np.zeros((G, d), np.uint16)
    for g in range(G):
        q[g, chans[g]] = f2bf(vals[g])
    S = orc.unit_scores(q, K, SCALE)
    Kf = bf2f(K).astype(np.float64)
    for j in range(n):
        exp = max(SCALE * vals[g] * Kf[j, chans[g]] for g in range(G))
        assert S[j] == exp, (j, S[j], exp)


def pin_scores_integer(orc):
    """Integer keys and constant queries: q_g = (g+1) * ones, so the logit of
    head g is scale*(g+1)*rowsum(K_j); the max picks g=G-1 for positive row
    sums and g=0 for negative ones."""
    rng = np.random.default_rng(2)
    G, d, n = 3, 32, 40
    K = f2bf(rng.integers(-3, 4, size=(n, d)).astype(np.float32))
    q = np.stack([f2bf(np.full(d, g + 1.0)) for g in range(G)])
    S = orc.unit_scores(q, K, 0.5)
    rs = bf2f(K).astype(np.float64).sum(axis=1)
    for j in range(n):
        mult = G if rs[j] > 0 else 1
        assert S[j] == 0.5 * mult * rs[j], (j, S[j], rs[j])


def pin_scores_batch_layout(orc):
    """Batch layout: query head q belongs to KV head q // G, keys of (b, h)
    start at ((b*Hkv + h)*max_ctx)*row_stride, padding columns of a strided row
    are never read, positions >= n_b score -inf."""
    rng = np.random.default_rng(3)
    B, Hq, Hkv, d, nmax, stride = 2, 8, 2, 16, 12, 20
    G = Hq // Hkv
    lens = np.array([9, 5], np.int32)
    keys = rand_bf(rng, (B, Hkv, nmax, stride))
    keys[..., d:] = 0x7FC0                    # NaN in the padding columns
    q = np.zeros((B, Hq, d), np.uint16)
    val = {}
    for b in range(B):
        for hq in range(Hq):
            c = (3 * hq + b) % d
            v = float(1 + hq + 10 * b)
            q[b, hq, c] = f2bf(v)
            val[(b, hq)] = (c, v)
    s = orc.shape(B, Hq, Hkv, d, nmax, key_row_stride=stride)
    S = orc.score_keys(s, q, keys, lens, SCALE)
    Kf = bf2f(keys).astype(np.float64)
    for b in range(B):
        for h in range(Hkv):
            for j in range(nmax):
                if j >= lens[b]:
                    assert S[b, h, j] == -math.inf
                    continue
                exp = max(SCALE * val[(b, hq)][1] * Kf[b, h, j, val[(b, hq)][0]]
                          for hq in range(h * G, h * G + G))
                assert S[b, h, j] == exp, (b, h, j, S[b, h, j], exp)


# --- selection ----------------------------------------------------------------
def _dominates(S, sub, n):
    """Definition of the critical set: every chosen position beats every
    unchosen one, by larger score, or by lower position on equal scores."""
    chosen = set(sub)
    for i in chosen:
        for u in range(n):
            if u in chosen:
                continue
            if not (S[i] > S[u] or (S[i] == S[u] and i < u)):
                return False
    return True


def pin_select_bruteforce(orc):
    """Enumerate every subset of size min(k, n) for n <= 10; exactly one obeys
    the definition and it is the oracle's, listed ascending, padded with -1."""
    rng = np.random.default_rng(4)
    levels = np.array([-1.5, 0.0, 0.25, 2.0, 7.0])
    for trial in range(250):
        n = int(rng.integers(0, 11))
        k = int(rng.integers(1, 13))
        if trial % 2:
            S = rng.choice(levels, size=n)           # many exact ties
        else:
            S = rng.standard_normal(n)
        idx, m = orc.unit_select(S, k)
        m_exp = min(k, n)
        assert m == m_exp, (n, k, m)
        valid = [c for c in itertools.combinations(range(n), m_exp)
                 if _dominates(S, c, n)]
        assert len(valid) == 1, (S, k, valid)
        assert list(idx[:m]) == list(valid[0]), (S, k, idx, valid)
        assert all(idx[m:] == -1), idx


def pin_select_reversal(orc):
    """Reversing the positions of distinct scores reverses the chosen set."""
    rng = np.random.default_rng(5)
    S = rng.standard_normal(200)
    idx, m = orc.unit_select(S, 37)
    idx_r, m_r = orc.unit_select(S[::-1].copy(), 37)
    assert m == m_r == 37
    assert sorted(199 - idx[:m]) == list(idx_r[:m])


def pin_select_small_contexts(orc):
    """n <= k selects every position; n = 0 selects none."""
    S = np.array([3.0, -1.0, 3.0, 0.5, 9.0])
    idx, m = orc.unit_select(S, 8)
    assert m == 5 and list(idx) == [0, 1, 2, 3, 4, -1, -1, -1]
    idx, m = orc.unit_select(np.zeros(0), 4)
    assert m == 0 and list(idx) == [-1] * 4


def pin_select_planted(orc, seeds=range(20)):
    """Tiny workload: the 16 keys planted at 4x the group's mean query
    direction are always among the 256 selected per KV head."""
    w = synth.WORKLOADS["tiny"]
    for seed in seeds:
        t = synth.make_layer(w, seed=seed)
        s = orc.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
        scores = orc.score_keys(s, synth.to_u16(t["q"]), synth.to_u16(t["k"]),
                                t["ctx_lens"].numpy(), SCALE, nthreads=2)
        idx, n_sel = orc.select_topk(s, scores, t["ctx_lens"].numpy(), w.k)
        marked = t["marked"].numpy()
        for b in range(w.batch):
            for h in range(w.kv_heads):
                planted = set(np.nonzero(marked[b, h])[0].tolist())
                assert len(planted) == 16
                assert planted <= set(idx[b, h, :n_sel[b, h]].tolist()), (seed, b, h)


# --- attention ----------------------------------------------------------------
def _sdpa(qf, kf, vf, scale):
    """torch's scaled-dot-product attention in float64 on the CPU."""
    q = torch.from_numpy(qf)[:, None, :]                    # [G][1][d]
    k = torch.from_numpy(kf)[None].expand(qf.shape[0], -1, -1).contiguous()
    v = torch.from_numpy(vf)[None].expand(qf.shape[0], -1, -1).contiguous()
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale)
    return o[:, 0, :].numpy()


def pin_attn_dense_library(orc):
    """With every row selected, the result is ordinary dense softmax attention
    (torch SDPA in float64)."""
    rng = np.random.default_rng(6)
    G, d, m = 4, 128, 300
    q, K, V = rand_bf(rng, (G, d)), rand_bf(rng, (m, d)), rand_bf(rng, (m, d))
    out, _ = orc.unit_attn(q, K, V, SCALE)
    ref = _sdpa(bf2f(q).astype(np.float64), bf2f(K).astype(np.float64),
                bf2f(V).astype(np.float64), SCALE)
    assert np.max(np.abs(out - ref)) < 1e-12, np.max(np.abs(out - ref))


def pin_attn_single_row(orc):
    """One selected row: its weight is exactly 1, so out is that V row."""
    rng = np.random.default_rng(7)
    q, K, V = rand_bf(rng, (4, 128)), rand_bf(rng, (1, 128)), rand_bf(rng, (1, 128))
    out, p = orc.unit_attn(q, K, V, SCALE)
    assert np.all(p == 1.0)
    assert np.array_equal(out, np.broadcast_to(bf2f(V[0]).astype(np.float64), out.shape))


def pin_attn_zero_query(orc):
    """A zero query gives equal logits: out is the mean of the V rows."""
    rng = np.random.default_rng(8)
    q = np.zeros((2, 128), np.uint16)
    K, V = rand_bf(rng, (50, 128)), rand_bf(rng, (50, 128))
    out, _ = orc.unit_attn(q, K, V, SCALE)
    mean = bf2f(V).astype(np.float64).mean(axis=0)
    assert np.max(np.abs(out - mean)) < 1e-13


def pin_attn_two_rows(orc):
    """Two rows with logits a and b: weights are the logistic function of the
    logit difference."""
    rng = np.random.default_rng(9)
    d = 128
    q = np.zeros((1, d), np.uint16)
    q[0, 17] = f2bf(1.0)
    K = rand_bf(rng, (2, d))
    K[0, 17], K[1, 17] = f2bf(1.25), f2bf(-0.5)
    V = rand_bf(rng, (2, d))
    out, _ = orc.unit_attn(q, K, V, 1.0)
    a, b = 1.25, -0.5
    w0 = 1.0 / (1.0 + math.exp(b - a))
    w1 = 1.0 / (1.0 + math.exp(a - b))
    Vf = bf2f(V).astype(np.float64)
    assert np.max(np.abs(out[0] - (w0 * Vf[0] + w1 * Vf[1]))) < 1e-14


def pin_attn_weights_normalised(orc):
    """Softmax weights are non-negative and sum to 1; V = 1 gives out = 1."""
    rng = np.random.default_rng(10)
    q, K = rand_bf(rng, (4, 128), 3.0), rand_bf(rng, (77, 128))
    V = np.full((77, 128), f2bf(1.0), np.uint16)
    out, p = orc.unit_attn(q, K, V, SCALE)
    assert np.all(p >= 0)
    assert np.max(np.abs(p.sum(axis=1) - 1.0)) < 1e-13
    assert np.max(np.abs(out - 1.0)) < 1e-13


def pin_attn_permutation(orc):
    """The result does not depend on the order of the selected rows."""
    rng = np.random.default_rng(11)
    q, K, V = rand_bf(rng, (4, 128)), rand_bf(rng, (90, 128)), rand_bf(rng, (90, 128))
    out, _ = orc.unit_attn(q, K, V, SCALE)
    perm = rng.permutation(90)
    out_p, _ = orc.unit_attn(q, K[perm], V[perm], SCALE)
    assert np.max(np.abs(out - out_p)) < 1e-12


def pin_attn_large_logits(orc):
    """Logits 2048 and 2040 (exp overflows fp64 without a max shift): the
    result is still the logistic mix of the two rows."""
    rng = np.random.default_rng(12)
    d = 128
    q = np.zeros((1, d), np.uint16)
    q[0, 3] = f2bf(1.0)
    K = rand_bf(rng, (2, d))
    K[0, 3], K[1, 3] = f2bf(2048.0), f2bf(2040.0)
    V = rand_bf(rng, (2, d))
    out, _ = orc.unit_attn(q, K, V, 1.0)
    w0 = 1.0 / (1.0 + math.exp(-8.0))
    Vf = bf2f(V).astype(np.float64)
    ref = w0 * Vf[0] + (1 - w0) * Vf[1]
    assert np.all(np.isfinite(out)) and np.max(np.abs(out[0] - ref)) < 1e-14


# --- gather ---------------------------------------------------------------------
def pin_gather_exact(orc):
    """Gather is an exact copy of the indexed rows (K|V interleaved source,
    row stride 2d); slots at or beyond n_sel are left untouched."""
    rng = np.random.default_rng(13)
    B, Hkv, nmax, d, k = 2, 3, 10, 8, 4
    src = rng.integers(0, 65536, size=(B, Hkv, nmax, 2, d)).astype(np.uint16)
    flat = src.reshape(-1)
    idx = np.full((B, Hkv, k), -1, np.int32)
    n_sel = rng.integers(0, k + 1, size=(B, Hkv)).astype(np.int32)
    for b in range(B):
        for h in range(Hkv):
            idx[b, h, :n_sel[b, h]] = np.sort(rng.choice(nmax, n_sel[b, h], replace=False))
    kd = np.full((B, Hkv, k, d), 0xABCD, np.uint16)
    vd = np.full((B, Hkv, k, d), 0xABCD, np.uint16)
    s = orc.shape(B, Hkv, Hkv, d, nmax, kv_row_stride=2 * d)
    orc.gather_kv(s, flat, flat[d:], idx, n_sel, k, kd, vd)
    for b in range(B):
        for h in range(Hkv):
            m = n_sel[b, h]
            assert np.array_equal(kd[b, h, :m], src[b, h, idx[b, h, :m], 0])
            assert np.array_equal(vd[b, h, :m], src[b, h, idx[b, h, :m], 1])
            assert np.all(kd[b, h, m:] == 0xABCD) and np.all(vd[b, h, m:] == 0xABCD)


# --- composition ------------------------------------------------------------------
def pin_pipeline_composition(orc):
    """The fused oracle equals score -> select -> gather -> attend, each part
    pinned above; with a separate selecting query, selection follows q_sel
    and attention follows q_att.  A budget >= n_b reduces to dense attention."""
    rng = np.random.default_rng(14)
    B, Hq, Hkv, d, nmax, k = 2, 8, 2, 128, 300, 40
    G = Hq // Hkv
    lens = np.array([300, 123], np.int32)
    q1, q2 = rand_bf(rng, (B, Hq, d)), rand_bf(rng, (B, Hq, d))
    K, V = rand_bf(rng, (B, Hkv, nmax, d)), rand_bf(rng, (B, Hkv, nmax, d))
    s = orc.shape(B, Hq, Hkv, d, nmax)
    for qs in (None, q2):
        idx, n_sel, out = orc.critical_kv_attn(s, q1, qs, K, K, V, lens, k, SCALE)
        sc = orc.score_keys(s, q1 if qs is None else qs, K, lens, SCALE)
        idx2, n_sel2 = orc.select_topk(s, sc, lens, k)
        assert np.array_equal(idx, idx2) and np.array_equal(n_sel, n_sel2)
        kb = np.zeros((B, Hkv, k, d), np.uint16)
        vb = np.zeros((B, Hkv, k, d), np.uint16)
        orc.gather_kv(s, K, V, idx, n_sel, k, kb, vb)
        out2 = orc.sparse_decode_attn(s, q1, kb, vb, n_sel, k, SCALE)
        assert np.max(np.abs(out - out2)) < 1e-12
    # q_sel != q_att really changes the set here (else the check above is void)
    idx_a, _, _ = orc.critical_kv_attn(s, q1, None, K, K, V, lens, k, SCALE)
    idx_b, _, _ = orc.critical_kv_attn(s, q1, q2, K, K, V, lens, k, SCALE)
    assert not np.array_equal(idx_a, idx_b)
    kbig = 512
    idx, n_sel, out = orc.critical_kv_attn(s, q1, q2, K, K, V, lens, kbig, SCALE)
    for b in range(B):
        for h in range(Hkv):
            n = lens[b]
            assert n_sel[b, h] == n and list(idx[b, h, :n]) == list(range(n))
            ref = _sdpa(bf2f(q1[b, h * G:(h + 1) * G]).astype(np.float64),
                        bf2f(K[b, h, :n]).astype(np.float64),
                        bf2f(V[b, h, :n]).astype(np.float64), SCALE)
            assert np.max(np.abs(out[b, h * G:(h + 1) * G] - ref)) < 1e-12


def pin_empty_context(orc):
    """n_b = 0: nothing selected, idx all -1, output zero."""
    rng = np.random.default_rng(15)
    B, Hq, Hkv, d, nmax, k = 2, 4, 1, 128, 16, 8
    lens = np.array([0, 5], np.int32)
    q = rand_bf(rng, (B, Hq, d))
    K, V = rand_bf(rng, (B, Hkv, nmax, d)), rand_bf(rng, (B, Hkv, nmax, d))
    s = orc.shape(B, Hq, Hkv, d, nmax)
    idx, n_sel, out = orc.critical_kv_attn(s, q, None, K, K, V, lens, k, SCALE)
    assert n_sel[0, 0] == 0 and np.all(idx[0, 0] == -1) and np.all(out[0] == 0.0)
    assert n_sel[1, 0] == 5 and list(idx[1, 0]) == [0, 1, 2, 3, 4, -1, -1, -1]


# --- chunk landmarks ------------------------------------------------------------
def pin_bf16_rounding(orc):
    """fp64 -> bf16: torch's fp32 -> bf16 conversion (round to nearest even) on
    fp32-representable values, closed-form midpoints, a value that rounding via
    fp32 would get wrong, and every finite bf16 pattern mapping to itself."""
    rng = np.random.default_rng(21)
    xs = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-30, 30, 4000),
                         [0.0, -0.0, 1.0, -1.0, 3.0e38, 1e-40, -7e-39]]).astype(np.float32)
    want = torch.from_numpy(xs).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    for x, w in zip(xs, want):
        assert orc.f64_to_bf16(float(x)) == int(w), (float(x), hex(int(w)))
    # 1 + 2^-8 lies halfway between 1 (even) and 1 + 2^-7: even wins; just above
    # it rounds up, which an intermediate fp32 rounding (to 1 + 2^-8) would lose
    assert orc.f64_to_bf16(1.0 + 2.0 ** -8) == 0x3F80
    assert orc.f64_to_bf16(1.0 + 2.0 ** -8 + 2.0 ** -40) == 0x3F81
    assert orc.f64_to_bf16(1.0 + 3 * 2.0 ** -8) == 0x3F82  # between 0x3F81 and 0x3F82
    assert orc.f64_to_bf16(-(1.0 + 3 * 2.0 ** -8)) == 0xBF82
    for b in range(0x10000):
        if (b & 0x7F80) == 0x7F80:  # inf / nan
            continue
        assert orc.f64_to_bf16(orc.bf16_to_f64(b)) == (b if b != 0x8000 else 0x8000), hex(b)


def pin_landmarks_unit_chunk(orc):
    """Chunks of one row: the landmarks are the keys, bit for bit (strided
    rows, ragged contexts; rows past n_b are not written)."""
    rng = np.random.default_rng(22)
    B, Hkv, n, d, stride = 2, 3, 13, 128, 136
    keys = rand_bf(rng, (B, Hkv, n, stride))
    lens = np.array([13, 9], np.int32)
    s = orc.shape(B, 2 * Hkv, Hkv, d, n, key_row_stride=stride)
    lm = orc.chunk_landmarks(s, 1, keys, lens, fill=0x7777)
    for b in range(B):
        nb = lens[b]
        assert np.array_equal(lm[b, :, :nb], keys[b, :, :nb, :d])
        assert np.all(lm[b, :, nb:] == 0x7777)


def pin_landmarks_closed_form(orc):
    """Means that bf16 holds exactly, and a partial last chunk that averages
    only the rows below n_b (the rows past it are huge, so counting them
    shows)."""
    d, C = 128, 4
    rows = np.zeros((1, 1, 12, d), np.float32)
    rows[0, 0, 0:4] = np.array([1.0, 2.0, 3.0, 4.0])[:, None]      # mean 2.5
    rows[0, 0, 4:8] = np.array([0.5, 0.25, -0.5, -0.25])[:, None]  # mean 0
    rows[0, 0, 4:8, 7] = [0.5, 0.25, 0.5, 0.25]                    # channel 7: 0.375
    rows[0, 0, 8:10] = np.array([-6.0, 2.0])[:, None]              # partial: -2
    rows[0, 0, 10:12] = 1e30
    keys = f2bf(rows)
    s = orc.shape(1, 1, 1, d, 12)
    lm = bf2f(orc.chunk_landmarks(s, C, keys, np.array([10], np.int32)))
    assert np.all(lm[0, 0, 0] == 2.5)
    assert lm[0, 0, 1, 7] == 0.375 and np.all(np.delete(lm[0, 0, 1], 7) == 0.0)
    assert np.all(lm[0, 0, 2] == -2.0)


def pin_landmarks_rounding(orc):
    """Means on a bf16 midpoint round to the even neighbour."""
    d = 128
    a, b, c = 1.0, 1.0 + 2.0 ** -7, 1.0 + 2.0 ** -6
    keys = f2bf(np.array([a, b, b, c], np.float32)[None, None, :, None] *
                np.ones((1, 1, 4, d), np.float32))
    lm = orc.chunk_landmarks(orc.shape(1, 1, 1, d, 4), 2, keys, np.array([4], np.int32))
    assert np.all(lm[0, 0, 0] == 0x3F80)  # (1 + (1+2^-7)) / 2: tie, even is 1.0
    assert np.all(lm[0, 0, 1] == 0x3F82)  # ((1+2^-7) + (1+2^-6)) / 2: tie, even up


def pin_expand_chunks(orc):
    rows, r = orc.expand_chunks(4, [0, 2], 10, 16)
    assert r == 6 and list(rows) == [0, 1, 2, 3, 8, 9] + [-1] * 10
    rows, r = orc.expand_chunks(3, [1, 2, 4], 100, 9)
    assert r == 9 and list(rows) == [3, 4, 5, 6, 7, 8, 12, 13, 14]
    rows, r = orc.expand_chunks(5, [], 7, 5)
    assert r == 0 and list(rows) == [-1] * 5


def pin_select_chunks_unit_chunk(orc):
    """Chunk size 1 is the per-position selection."""
    rng = np.random.default_rng(23)
    B, Hq, Hkv, n, d, k = 2, 8, 2, 300, 128, 32
    keys = rand_bf(rng, (B, Hkv, n, d))
    q = rand_bf(rng, (B, Hq, d))
    lens = np.array([300, 77], np.int32)
    s = orc.shape(B, Hq, Hkv, d, n)
    lm = orc.chunk_landmarks(s, 1, keys, lens)
    cidx, nch, rows, nrows = orc.select_chunks(s, 1, q, lm, lens, k, SCALE)
    idx, nsel = orc.select_topk(s, orc.score_keys(s, q, keys, lens, SCALE), lens, k)
    assert np.array_equal(cidx, idx) and np.array_equal(rows, idx)
    assert np.array_equal(nch, nsel) and np.array_equal(nrows, nsel)


def pin_select_chunks_bruteforce(orc):
    """Tiny contexts: the chosen chunks are the unique subset of size kc whose
    scores (numpy dot products with the landmarks, max over the group) all beat
    the others, ties to the lower chunk; rows are those chunks' rows below n."""
    rng = np.random.default_rng(24)
    d, G, C, k = 128, 2, 3, 6
    for trial in range(30):
        n = int(rng.integers(4, 13))
        keys = rand_bf(rng, (1, 1, 12, d))
        if trial % 3 == 0:  # exact ties between chunks
            keys[0, 0, 3:6] = keys[0, 0, 0:3]
        q = rand_bf(rng, (1, G, d))
        s = orc.shape(1, G, 1, d, 12)
        lm = orc.chunk_landmarks(s, C, keys, np.array([n], np.int32))
        nc = (n + C - 1) // C
        L = bf2f(lm[0, 0, :nc]).astype(np.float64)
        S = (bf2f(q[0]).astype(np.float64) @ L.T).max(axis=0) * SCALE
        kc = min(k // C, nc)
        best = None
        for sub in itertools.combinations(range(nc), kc):
            if _dominates(S, sub, nc):
                best = sub
                break
        cidx, nch, rows, nrows = orc.select_chunks(s, C, q, lm, np.array([n], np.int32), k,
                                                   SCALE)
        assert nch[0, 0] == kc and tuple(cidx[0, 0, :kc]) == best, (trial, best, cidx)
        want = [c * C + t for c in best for t in range(C) if c * C + t < n]
        assert nrows[0, 0] == len(want) and list(rows[0, 0, :len(want)]) == want


# --- dual-token attention ---------------------------------------------------------
def _dual_case(rng, B=2, Hq=8, Hkv=2, k=24, m=(17, 0), d=128):
    s_shape = dict(B=B, Hq=Hq, Hkv=Hkv, d=d, k=k)
    kb = rand_bf(rng, (B, Hkv, k, d))
    vb = rand_bf(rng, (B, Hkv, k, d))
    kl = rand_bf(rng, (B, Hkv, 2, d))
    vl = rand_bf(rng, (B, Hkv, 2, d))
    qc = rand_bf(rng, (B, Hq, d))
    qs = rand_bf(rng, (B, Hq, d))
    n_sel = np.array([[m[b % len(m)]] * Hkv for b in range(B)], np.int32)
    return s_shape, qc, qs, kb, vb, n_sel, kl, vl


def pin_dual_token_causal_sdpa(orc):
    """Both tokens against torch's scaled_dot_product_attention in fp64 on the
    dense sequence [selected rows, T_i, T'_{i+1}] with the causal mask on the
    two new positions."""
    rng = np.random.default_rng(31)
    sh, qc, qs, kb, vb, n_sel, kl, vl = _dual_case(rng)
    B, Hq, Hkv, d, k = sh["B"], sh["Hq"], sh["Hkv"], sh["d"], sh["k"]
    s = orc.shape(B, Hq, Hkv, d, 64)
    oc, os_ = orc.dual_token_attn(s, qc, qs, kb, vb, n_sel, kl, vl, k, SCALE)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            m = int(n_sel[b, h])
            K = torch.from_numpy(np.concatenate([bf2f(kb[b, h, :m]), bf2f(kl[b, h])]).astype(np.float64))
            V = torch.from_numpy(np.concatenate([bf2f(vb[b, h, :m]), bf2f(vl[b, h])]).astype(np.float64))
            Q = torch.from_numpy(np.stack([bf2f(qc[b, h * G:(h + 1) * G]),
                                           bf2f(qs[b, h * G:(h + 1) * G])]).astype(np.float64))
            mask = torch.ones(2, 1, m + 2, dtype=torch.bool)
            mask[0, 0, m + 1] = False  # the current token does not see the speculative one
            ref = torch.nn.functional.scaled_dot_product_attention(
                Q, K[None].expand(2, -1, -1), V[None].expand(2, -1, -1), attn_mask=mask,
                scale=SCALE).numpy()
            assert np.abs(oc[b, h * G:(h + 1) * G] - ref[0]).max() < 1e-12
            assert np.abs(os_[b, h * G:(h + 1) * G] - ref[1]).max() < 1e-12


def pin_dual_token_empty_set(orc):
    """No selected rows: the current token sees only itself (its V row,
    exactly); the speculative token sees the two new rows (logistic weights)."""
    rng = np.random.default_rng(32)
    sh, qc, qs, kb, vb, n_sel, kl, vl = _dual_case(rng, B=1, m=(0,))
    B, Hq, Hkv, d, k = sh["B"], sh["Hq"], sh["Hkv"], sh["d"], sh["k"]
    oc, os_ = orc.dual_token_attn(orc.shape(B, Hq, Hkv, d, 64), qc, qs, kb, vb, n_sel, kl, vl,
                                  k, SCALE)
    G = Hq // Hkv
    for h in range(Hkv):
        v0, v1 = bf2f(vl[0, h, 0]).astype(np.float64), bf2f(vl[0, h, 1]).astype(np.float64)
        k0, k1 = bf2f(kl[0, h, 0]).astype(np.float64), bf2f(kl[0, h, 1]).astype(np.float64)
        for g in range(G):
            assert np.array_equal(oc[0, h * G + g], v0)
            q = bf2f(qs[0, h * G + g]).astype(np.float64)
            p1 = 1.0 / (1.0 + math.exp(SCALE * (q @ k0 - q @ k1)))
            assert np.abs(os_[0, h * G + g] - ((1 - p1) * v0 + p1 * v1)).max() < 1e-12


def pin_dual_token_mask_invariance(orc):
    """Changing the speculative token's row never changes the current token's
    output, and does change the speculative token's."""
    rng = np.random.default_rng(33)
    sh, qc, qs, kb, vb, n_sel, kl, vl = _dual_case(rng)
    B, Hq, Hkv, d, k = sh["B"], sh["Hq"], sh["Hkv"], sh["d"], sh["k"]
    s = orc.shape(B, Hq, Hkv, d, 64)
    oc1, os1 = orc.dual_token_attn(s, qc, qs, kb, vb, n_sel, kl, vl, k, SCALE)
    kl2, vl2 = kl.copy(), vl.copy()
    kl2[:, :, 1] = rand_bf(rng, kl2[:, :, 1].shape, scale=8.0)
    vl2[:, :, 1] = rand_bf(rng, vl2[:, :, 1].shape, scale=8.0)
    oc2, os2 = orc.dual_token_attn(s, qc, qs, kb, vb, n_sel, kl2, vl2, k, SCALE)
    assert np.array_equal(oc1, oc2)
    assert np.abs(os1 - os2).max() > 1e-3


# --- low-rank key reconstruction ---------------------------------------------------
def pin_reconstruct_identity(orc):
    """rank = d and W = I: the reconstruction is the U row itself, bit for bit
    (slots past n_sel untouched)."""
    rng = np.random.default_rng(41)
    B, Hkv, n, d, k = 2, 2, 40, 128, 8
    U = rand_bf(rng, (B, Hkv, n, d))
    W = np.tile(f2bf(np.eye(d, dtype=np.float32)), (B, Hkv, 1, 1))
    idx = rng.integers(0, n, size=(B, Hkv, k)).astype(np.int32)
    nsel = np.array([[8, 3], [0, 5]], np.int32)
    out = orc.reconstruct_keys(orc.shape(B, 2 * Hkv, Hkv, d, n), d, U, W, idx, nsel, k)
    for b in range(B):
        for h in range(Hkv):
            m = nsel[b, h]
            assert np.array_equal(out[b, h, :m], U[b, h, idx[b, h, :m]])
            assert np.all(out[b, h, m:] == 0x7777)


def pin_reconstruct_library(orc):
    """Small exact factors (values in multiples of 1/8, rank 4): the products
    and sums are exact in fp64 and fit bf16, so the result equals numpy's
    matrix product, rounded by torch to bf16 (a no-op here)."""
    rng = np.random.default_rng(42)
    B, Hkv, n, d, r, k = 1, 3, 20, 128, 4, 6
    U = f2bf(rng.integers(-8, 9, size=(B, Hkv, n, r)).astype(np.float32) / 8)
    W = f2bf(rng.integers(-4, 5, size=(B, Hkv, r, d)).astype(np.float32) / 4)
    idx = np.stack([[rng.permutation(n)[:k] for _ in range(Hkv)]]).astype(np.int32)
    nsel = np.full((B, Hkv), k, np.int32)
    out = orc.reconstruct_keys(orc.shape(B, Hkv, Hkv, d, n), r, U, W, idx, nsel, k)
    for h in range(Hkv):
        ref = bf2f(U[0, h, idx[0, h]]).astype(np.float64) @ bf2f(W[0, h]).astype(np.float64)
        want = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).view(torch.int16)
        assert np.array_equal(out[0, h].view(np.int16), want.numpy())


def pin_reconstruct_rounding(orc):
    """A sum landing on a bf16 midpoint rounds to even: 1 + 2^-8 from two
    rank terms (1 and 2^-8) gives 1.0; 1 + 2^-8 + 2^-16 gives 1 + 2^-7."""
    d = 128
    U = f2bf(np.array([[[[1.0, 2.0 ** -8, 2.0 ** -16]]]], np.float32))
    W1 = f2bf(np.concatenate([np.ones((1, 1, 2, d)), np.zeros((1, 1, 1, d))], axis=2)
              .astype(np.float32))
    W2 = f2bf(np.ones((1, 1, 3, d), np.float32))
    s = orc.shape(1, 1, 1, d, 1)
    idx, nsel = np.zeros((1, 1, 1), np.int32), np.ones((1, 1), np.int32)
    assert np.all(orc.reconstruct_keys(s, 3, U, W1, idx, nsel, 1) == 0x3F80)
    assert np.all(orc.reconstruct_keys(s, 3, U, W2, idx, nsel, 1) == 0x3F81)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
