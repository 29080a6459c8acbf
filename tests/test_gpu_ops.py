"""Single-kernel parity on the GPU: streaming GEMM, tree attention, LM-head
reductions, tree truncation and acceptance, each against the oracle's definition
on the same seeded inputs, including the full 7B and large-model shapes."""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import mask_words, need_gpu, note, seeded, to_np

pytestmark = pytest.mark.gpu

GEMM_CASES = [
    # dtype, M, N, K, sampled
    ("f32", 1, 256, 256, False), ("f32", 41, 768, 256, False), ("f32", 41, 256, 688, False),
    ("f32", 41, 1376, 256, False), ("f32", 130, 512, 256, False), ("f32", 16, 1024, 256, False),
    ("bf16", 1, 4096, 4096, False), ("bf16", 8, 4096, 4096, False), ("bf16", 32, 8192, 4096, False),
    ("bf16", 64, 12288, 4096, False), ("bf16", 64, 4096, 4096, False), ("bf16", 64, 4096, 11008, False),
    ("bf16", 64, 22016, 4096, False), ("bf16", 64, 125696, 4096, True), ("bf16", 64, 10240, 8192, False),
    ("bf16", 64, 8192, 28672, True), ("bf16", 512, 4096, 4096, True), ("bf16", 100, 1024, 512, False),
    ("bf16", 3, 48, 64, False),
    # streaming kernel with one 128-row chunk (65..128 rows): 7B shapes and ragged row counts
    ("bf16", 128, 12288, 4096, True), ("bf16", 128, 4096, 11008, True), ("bf16", 128, 22016, 4096, True),
    ("bf16", 65, 4096, 4096, False), ("bf16", 127, 125696, 4096, True),
    # register-blocked kernel: swept 7B shapes, the default rule, ragged row counts
    ("bf16", 129, 12288, 4096, True), ("bf16", 256, 4096, 11008, True), ("bf16", 300, 4096, 4096, True),
    ("bf16", 512, 22016, 4096, True), ("bf16", 200, 125696, 4096, True), ("bf16", 130, 1024, 512, False),
    # the cost surface's largest cells: 1024 and 2048 verify rows (batch 16 x 64- and 128-token trees)
    ("bf16", 1024, 12288, 4096, True), ("bf16", 1024, 4096, 4096, False), ("bf16", 1024, 22016, 4096, True),
    ("bf16", 1024, 4096, 11008, True), ("bf16", 1024, 125696, 4096, True),
    ("bf16", 2048, 12288, 4096, True), ("bf16", 2048, 4096, 4096, True), ("bf16", 2048, 22016, 4096, True),
    ("bf16", 2048, 4096, 11008, True), ("bf16", 2048, 125696, 4096, True), ("bf16", 1500, 4096, 4096, True),
    # 32x32 matrix-core kernel: the 7B output and down projections at 512 rows (4 K splits),
    # ragged rows
    ("bf16", 512, 4096, 11008, True), ("bf16", 520, 4096, 11008, True), ("bf16", 700, 4096, 4096, False),
    # the cost surface's batch-48 cells: 3072 and 6144 verify rows (48 x 64- and 128-token trees)
    ("bf16", 3072, 12288, 4096, True), ("bf16", 6144, 12288, 4096, True), ("bf16", 6144, 4096, 4096, True),
    ("bf16", 6144, 4096, 11008, True), ("bf16", 6144, 22016, 4096, True), ("bf16", 6144, 125696, 4096, True),
]


@pytest.mark.parametrize("dt,M,N,K,sampled", GEMM_CASES)
def test_linear_matches_definition(dt, M, N, K, sampled):
    P = need_gpu()
    note(f"linear {dt} M={M} N={N} K={K}")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    X = seeded((M, K), 1000 + M, 1.0, tdt)
    W = seeded((N, K), 2000 + N, 0.02, tdt)
    Wp = P.pack_matrix(W)
    Yd = P.op_linear(X, Wp, N)
    torch.cuda.synchronize()
    cols, rows = np.arange(N), np.arange(M)
    if sampled:
        rng = np.random.default_rng(0)
        cols = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N), rng.choice(N, 512, replace=False)]))
        if M > 2048:  # first and last row tiles and a random sample between
            rows = np.unique(np.concatenate([np.arange(64), np.arange(M - 64, M), rng.choice(M, 256, replace=False)]))
    ri, ci = torch.as_tensor(rows, device=X.device), torch.as_tensor(cols, device=X.device)
    Y = to_np(Yd[ri][:, ci])
    Xn, Wn = to_np(X[ri]), to_np(W[ci])
    ref = Xn @ Wn.T
    bound = 1e-4 * (np.abs(Xn) @ np.abs(Wn).T) + 1e-7
    err = np.abs(Y - ref)
    assert np.all(err <= bound), float(np.max(err / bound))


SWIGLU_CASES = [
    # dtype, M, F, K, sampled: the 7B MLP at 64 rows (streaming), 300 and 1024 rows
    # (register-blocked), 512 rows (256-row matrix-core workgroups); ragged rows and a last
    # feature group with 4 of its 6 tile pairs past F on the matrix-core kernel; f32
    ("bf16", 64, 11008, 4096, True), ("bf16", 300, 11008, 4096, True), ("bf16", 512, 11008, 4096, True),
    ("bf16", 1024, 11008, 4096, True), ("bf16", 520, 1408, 512, False), ("bf16", 777, 1408, 512, False),
    ("f32", 41, 1376, 256, False), ("bf16", 6144, 11008, 4096, True),
]


@pytest.mark.parametrize("dt,M,F,K,sampled", SWIGLU_CASES)
def test_swiglu_matches_definition(dt, M, F, K, sampled):
    """The target layer's gated MLP activation against its definition in float64 on the same
    inputs: each product within the fp32-accumulation bound of the linear test, the result
    within one ulp of the storage type plus the products' errors carried through."""
    P = need_gpu()
    note(f"swiglu {dt} M={M} F={F} K={K}")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    X = seeded((M, K), 3000 + M, 1.0, tdt)
    Wg = seeded((F, K), 4000 + F, 0.02, tdt)
    Wu = seeded((F, K), 5000 + F, 0.02, tdt)
    actd = P.op_swiglu(X, P.pack_matrix(Wg), P.pack_matrix(Wu), F).float()
    torch.cuda.synchronize()
    cols, rows = np.arange(F), np.arange(M)
    if sampled:
        rng = np.random.default_rng(1)
        cols = np.unique(np.concatenate([np.arange(64), np.arange(F - 96, F), rng.choice(F, 384, replace=False)]))
        if M > 2048:
            rows = np.unique(np.concatenate([np.arange(256), np.arange(M - 256, M), rng.choice(M, 256, replace=False)]))
    idx, ri = torch.as_tensor(cols, device=Wg.device), torch.as_tensor(rows, device=Wg.device)
    act = to_np(actd[ri][:, idx])
    Xn, Gn, Un = to_np(X[ri]).astype(np.float64), to_np(Wg[idx]).astype(np.float64), to_np(Wu[idx]).astype(np.float64)
    g, u = Xn @ Gn.T, Xn @ Un.T
    ref = oracle.silu(g) * u
    dg, du = 1e-4 * (np.abs(Xn) @ np.abs(Gn).T), 1e-4 * (np.abs(Xn) @ np.abs(Un).T)
    ulp = 2.0 ** -7 if dt == "bf16" else 2.0 ** -22
    bound = ulp * np.abs(ref) + 1.1 * np.abs(u) * dg + np.abs(oracle.silu(g)) * du + 1e-7
    err = np.abs(act - ref)
    assert np.all(err <= bound), float(np.max(err / bound))


def test_linear_is_deterministic():
    P = need_gpu()
    note("linear determinism")
    X = seeded((64, 11008), 5, 1.0, torch.bfloat16)
    W = seeded((4096, 11008), 6, 0.02, torch.bfloat16)
    Wp = P.pack_matrix(W)
    a = P.op_linear(X, Wp, 4096)
    b = P.op_linear(X, Wp, 4096)
    assert torch.equal(a, b)


def _tree_parents(T, rng, depth_max=4):
    par = [-1]
    depth = [0]
    for i in range(1, T):
        cands = [j for j in range(i) if depth[j] < depth_max]
        p = int(rng.choice(cands))
        par.append(p)
        depth.append(depth[p] + 1)
    return par


ATT_CASES = [
    # dtype, L, T, Hq, Hkv, hd, causal
    ("f32", 128, 41, 4, 4, 64, False), ("f32", 0, 41, 4, 4, 64, True), ("f32", 37, 5, 2, 1, 32, False),
    ("f32", 200, 64, 4, 4, 64, True), ("bf16", 1024, 64, 8, 8, 128, False), ("bf16", 1, 1, 4, 4, 128, False),
    ("bf16", 3000, 64, 8, 1, 128, False), ("bf16", 77, 128, 4, 2, 64, False), ("bf16", 256, 256, 2, 2, 128, True),
    ("bf16", 4096, 64, 4, 4, 128, False),
    # the context sweep's longest cells and the largest context the kernel takes (65536 keys)
    ("bf16", 32768, 64, 8, 8, 128, False), ("bf16", 16384, 128, 8, 1, 128, False),
    ("bf16", 65472, 64, 2, 2, 128, False),
]


@pytest.mark.parametrize("dt,L,T,Hq,Hkv,hd,causal", ATT_CASES)
def test_tree_attention_matches_oracle(dt, L, T, Hq, Hkv, hd, causal):
    P = need_gpu()
    note(f"attention {dt} L={L} T={T} Hq={Hq} Hkv={Hkv} hd={hd} causal={causal}")
    if T > 128 and not causal:
        pytest.skip("trees are at most 128 tokens")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    rng = np.random.default_rng(L + T)
    Q = seeded((T, Hq, hd), 11 + L, 1.0, tdt)
    Kp = seeded((max(L, 1), Hkv, hd), 12 + L, 1.0, tdt)[:L]
    Vp = seeded((max(L, 1), Hkv, hd), 13 + L, 1.0, tdt)[:L]
    Kt = seeded((T, Hkv, hd), 14 + L, 1.0, tdt)
    Vt = seeded((T, Hkv, hd), 15 + L, 1.0, tdt)
    par = None if causal else _tree_parents(T, rng)
    if T > 128:
        # causal chunk longer than one tree: run as the prefill path does
        O = P.op_attention(Q, Kp, Vp, Kt, Vt, None, True)
    else:
        O = P.op_attention(Q, Kp, Vp, Kt, Vt, par, causal)
    torch.cuda.synchronize()
    vis_tail = np.tril(np.ones((T, T), dtype=bool)) if causal else oracle.tree_mask(par)
    vis = np.concatenate([np.ones((T, L), dtype=bool), vis_tail], axis=1)
    ref = oracle.attention(to_np(Q), np.concatenate([to_np(Kp), to_np(Kt)]),
                           np.concatenate([to_np(Vp), to_np(Vt)]), vis)
    tol = 1e-2 if dt == "bf16" else 2e-5
    err = np.max(np.abs(to_np(O) - ref))
    assert err < tol, err


def test_argmax_and_topk_exact():
    P = need_gpu()
    note("argmax/topk")
    M, V = 40, 125696
    logits = seeded((M, V), 21, 1.3)
    # planted exact ties: lower index must win
    logits[0, 100] = 50.0
    logits[0, 7] = 50.0
    logits[1, 5] = 40.0
    logits[1, 9] = 40.0
    logits[1, 3] = 40.0
    a = P.op_argmax(logits).cpu().numpy()
    L = logits.cpu().numpy()
    assert np.array_equal(a, np.argmax(L, axis=1))
    assert a[0] == 7 and a[1] == 3
    for k in (1, 2, 4, 8, 16):
        tok, logp = P.op_topk(logits, k)
        tok, logp = tok.cpu().numpy(), logp.cpu().numpy()
        for m in range(M):
            ids = oracle.topk_ids(L[m].astype(np.float64), k)
            assert list(tok[m]) == list(ids), (k, m)
            lse = oracle.logsumexp(L[m].astype(np.float64))
            assert np.max(np.abs(logp[m] - (L[m, ids] - lse))) < 2e-5


def _random_candidates(topk, rng, tie_every=0):
    depth, token, parent, lp = [0], [int(rng.integers(0, 1000))], [-1], [np.float32(0)]
    for j, k in enumerate(topk, start=1):
        for n in [i for i in range(len(depth)) if depth[i] == j - 1]:
            logp = -np.sort(rng.exponential(1.0, k)).astype(np.float32)
            if tie_every:
                logp = np.round(logp * 2) / 2  # many exact ties
            for t, l in zip(rng.choice(125696, k, replace=False), logp):
                depth.append(j); token.append(int(t)); parent.append(n)
                lp.append(np.float32(lp[n] + np.float32(l)))
    return (np.array(depth, np.int32), np.array(token, np.int32), np.array(parent, np.int32),
            np.array(lp, np.float32))


@pytest.mark.parametrize("topk,T,ties", [((4, 3, 2), 41, 0), ((8, 4, 2), 64, 0), ((8, 4, 2), 64, 1),
                                         ((8, 4, 2, 2), 64, 0), ((16, 4, 2), 128, 0), ((4, 2, 2), 16, 1),
                                         ((3,), 4, 0), ((2, 2, 2, 2, 2, 2), 100, 1)])
def test_tree_build_bit_exact(topk, T, ties):
    P = need_gpu()
    note(f"tree_build topk={topk} T={T}")
    rng = np.random.default_rng(T + len(topk) + ties)
    d, tok, par, lp = _random_candidates(topk, rng, ties)
    L = int(rng.integers(0, 5000))
    ref = oracle.build_tree(d, tok, par, lp, T, L)
    cu = lambda a: torch.as_tensor(a, device="cuda")
    out = P.op_tree_build(cu(tok), cu(par), cu(d), cu(lp), T, L)
    torch.cuda.synchronize()
    assert np.array_equal(out["tokens"].cpu().numpy(), ref.tokens)
    assert np.array_equal(out["parent"].cpu().numpy(), ref.parent)
    assert np.array_equal(out["depth"].cpu().numpy(), ref.depth)
    assert np.array_equal(out["pos"].cpu().numpy(), ref.pos)
    got_mask = out["mask"].cpu().numpy().view(np.uint64).reshape(T, -1)
    assert np.array_equal(got_mask, mask_words(ref.mask))


def test_acceptance_bit_exact():
    P = need_gpu()
    note("accept")
    rng = np.random.default_rng(3)
    for trial in range(60):
        T = int(rng.integers(1, 129))
        par = _tree_parents(T, rng, depth_max=4)
        tokens = [0] * T
        for p in range(T):
            kids = [c for c in range(T) if par[c] == p]
            for c, t in zip(kids, rng.choice(200, len(kids), replace=False)):
                tokens[c] = int(t)
        target = []
        for i in range(T):
            kids = [c for c in range(T) if par[c] == i]
            target.append(tokens[int(rng.choice(kids))] if kids and rng.random() < 0.8 else int(rng.integers(0, 200)))
        acc_ref, bonus_ref = oracle.accept(tokens, par, target)
        cu = lambda a: torch.as_tensor(np.asarray(a, np.int32), device="cuda")
        acc, acc_len, bonus = P.op_accept(cu(tokens), cu(par), cu(target), 4)
        A = int(acc_len.item())
        assert A == len(acc_ref)
        assert list(acc.cpu().numpy()[:A]) == acc_ref
        assert int(bonus.item()) == bonus_ref


def _slot_view(cache, block_table, n_slots, which_v):
    """Logical rows [slot][n_kv][hd] of a paged pool [blocks][n_kv][16*hd], read through the
    documented in-block layouts: K in score-fragment order (chunk d // KC, lane key + 16 *
    ((d % KC) // EPL), element d % EPL), V as [d // 16][key // 4][d % 16][key % 4]."""
    nb, nkv, per = cache.shape
    hd = per // 16
    EPL = 8 if cache.dtype == np.uint16 else 4
    KC = 4 * EPL
    d = np.arange(hd)
    out = np.empty((n_slots, nkv, hd), dtype=cache.dtype)
    for s in range(n_slots):
        blk, key = block_table[s // 16], s % 16
        if which_v:
            idx = (((d >> 4) * 4 + (key >> 2)) * 16 + (d & 15)) * 4 + (key & 3)
        else:
            idx = ((d // KC) * 64 + key + 16 * ((d % KC) // EPL)) * EPL + (d % EPL)
        out[s] = cache[blk][:, idx]
    return out


@pytest.mark.parametrize("dt,acc", [("bf16", [0, 5, 9, 17]), ("bf16", [0, 1, 3, 4]), ("bf16", [0, 2, 3]),
                                    ("bf16", [0]), ("f32", [0, 7, 8, 20, 31]), ("bf16", [0, 3, 12, 40, 63])])
def test_compact_moves_accepted_slots_bit_exactly(dt, acc):
    """KV compaction (the commit of Sec. 2.1): on every layer the rows of slot L + acc[j]
    land in slot L + j byte for byte, sources that are also destinations (acc[j'] = j) are
    read before being overwritten, and every other slot is left as it was.  The sequence's
    pages are scattered over the pool in a shuffled order, with L crossing a page."""
    P = need_gpu()
    note(f"compact {dt} acc={acc}")
    nl, nkv, hd, nb = 3, 2, 128 if dt == "bf16" else 64, 12
    rng = np.random.default_rng(len(acc) * 31 + acc[-1])
    table = rng.permutation(nb)[:7].astype(np.int32)
    L = 37
    np_dt = np.uint16 if dt == "bf16" else np.uint32
    k0 = rng.integers(0, 2 ** (16 if dt == "bf16" else 32), size=(nl, nb, nkv, 16 * hd), dtype=np.uint64).astype(np_dt)
    v0 = rng.integers(0, 2 ** (16 if dt == "bf16" else 32), size=(nl, nb, nkv, 16 * hd), dtype=np.uint64).astype(np_dt)
    tdt = torch.int16 if dt == "bf16" else torch.int32
    kc = torch.from_numpy(k0.view(np.int16 if dt == "bf16" else np.int32)).cuda()
    vc = torch.from_numpy(v0.view(np.int16 if dt == "bf16" else np.int32)).cuda()
    if dt == "bf16":
        kc, vc = kc.view(torch.bfloat16), vc.view(torch.bfloat16)
    else:
        kc, vc = kc.view(torch.float32), vc.view(torch.float32)
    P.op_compact(kc, vc, table, L, acc)
    k1 = kc.view(tdt).cpu().numpy().view(np_dt)
    v1 = vc.view(tdt).cpu().numpy().view(np_dt)
    n_slots = 16 * len(table)
    for layer in range(nl):
        for which, before, after in ((0, k0, k1), (1, v0, v1)):
            b = _slot_view(before[layer], table, n_slots, which)
            a = _slot_view(after[layer], table, n_slots, which)
            want = b.copy()
            want[L + np.arange(len(acc))] = b[L + np.asarray(acc)]  # gather all, then store
            assert np.array_equal(a, want), (layer, which)
        # blocks outside the table are untouched
        rest = np.setdiff1d(np.arange(nb), table)
        assert np.array_equal(k1[layer][rest], k0[layer][rest]) and np.array_equal(v1[layer][rest], v0[layer][rest])


def test_compact_rejects_out_of_range_arguments():
    P = need_gpu()
    note("compact argument checks")
    kc = torch.zeros(1, 4, 1, 16 * 32, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    for table, L, acc in (([0, 4], 0, [0]), ([0, 1], 31, [0, 1]), ([0, 1], 10, [0, -1]), ([0, 1], 0, [0] * 10)):
        with pytest.raises(P.CloverError):
            P.op_compact(kc, vc, table, L, acc)
    assert torch.count_nonzero(kc.float()) == 0

