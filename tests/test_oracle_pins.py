"""Pins of the CPU oracle against facts it does not compute itself.

Each test fixes one part of the layer (Mixture-of-Parallelisms Sec. 2.1: a
router sends each token to its top-k of E experts and the expert outputs are
combined with the router weights; Sec. 3.3: expert parallelism moves where
the work runs, never the result) to something independent of the oracle:
hand-derived IEEE values, library routines (numpy sort/bincount/matmul),
closed forms, algebraic identities and fp64 finite differences.
"""
import json
import os

import numpy as np
import pytest

import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def f32_to_bf16_bits(a):
    """Round float values to bf16 bits (RNE), for building tiny inputs."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def bits_to_f64(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def small_case(T=64, d=32, E=8, k=2, f=24, seed=0, E_loc=None, e_begin=0, bias=None):
    rng = np.random.default_rng(seed)
    E_loc = E if E_loc is None else E_loc
    x = f32_to_bf16_bits(rng.standard_normal((T, d)))
    w_r = (rng.standard_normal((d, E)) * 0.3).astype(np.float32)
    wg = f32_to_bf16_bits(rng.standard_normal((E_loc, d, f)) * 0.2)
    wu = f32_to_bf16_bits(rng.standard_normal((E_loc, d, f)) * 0.2)
    wd = f32_to_bf16_bits(rng.standard_normal((E_loc, f, d)) * 0.2)
    dy = f32_to_bf16_bits(rng.standard_normal((T, d)))
    return dict(x=x, w_r=w_r, bias=bias, wg=wg, wu=wu, wd=wd, dy=dy, k=k, E=E,
                E_loc=E_loc, e_begin=e_begin)


# ---------------------------------------------------------------- router
def test_logits_golden_chain(orc):
    g = json.load(open(os.path.join(GOLD, "router_chain.json")))
    for c in g["cases"]:
        x = f32_to_bf16_bits(np.array([c["x"]], dtype=np.float32))
        assert np.array_equal(bits_to_f64(x)[0], np.array(c["x"])), c["name"]
        w = np.array(c["w"], dtype=np.float32).reshape(-1, 1)
        b = None if c["bias"] is None else np.array([c["bias"]], dtype=np.float32)
        lg = orc.logits(x, w, b, "f32")
        assert lg.shape == (1, 1)
        assert float(lg[0, 0]) == c["expected_f32"], (c["name"], float(lg[0, 0]))
        if "expected_f32_hex" in c:
            assert hex(lg.view(np.uint32)[0, 0]) == c["expected_f32_hex"]
        if "expected_sign_bit" in c:
            assert (int(lg.view(np.uint32)[0, 0]) >> 31) == c["expected_sign_bit"]
        if "expected_exact" in c:
            assert float(orc.logits(x, w, b, "f64")[0, 0]) == c["expected_exact"]


def test_logits_match_fp64_matmul(orc):
    c = small_case(T=96, d=200, E=40, seed=3)
    bias = np.random.default_rng(1).standard_normal(40).astype(np.float32)
    lg = orc.logits(c["x"], c["w_r"], bias, "f32")
    ref = bits_to_f64(c["x"]) @ c["w_r"].astype(np.float64) + bias
    assert np.max(np.abs(lg - ref)) <= 1e-5 * np.max(np.abs(ref))
    lg64 = orc.logits(c["x"], c["w_r"], bias, "f64")
    assert np.max(np.abs(lg64 - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_topk_matches_lexsort(orc):
    rng = np.random.default_rng(5)
    T, E = 300, 24
    # coarse grid -> many exact ties, plus signed zeros
    lg = (np.round(rng.standard_normal((T, E)) * 2) / 2).astype(np.float32)
    lg[0, :] = 0.0
    lg[0, 3] = -0.0
    lg[1, :] = -1.0
    lg[1, :4] = [-0.0, 0.0, -0.0, 0.0]
    for k in (1, 3, E):
        idx, _ = orc.topk(lg, k)
        for t in range(T):
            # lexsort: last key is primary -> (-logit) primary, index secondary
            ref = np.lexsort((np.arange(E), -lg[t].astype(np.float64)))[:k]
            assert np.array_equal(idx[t], ref), (t, k)
    idx, _ = orc.topk(lg, 4)
    assert list(idx[0]) == [0, 1, 2, 3]          # all zero: lowest index first
    assert list(idx[1][:4]) == [0, 1, 2, 3]      # -0 == +0 is a tie


def test_topk_nan_ranks_as_minus_inf(orc):
    """NaN logits rank as -inf (ties by index): the selection always names
    valid experts.  Brute force: lexsort with NaN replaced by -inf."""
    E = 12
    lg = np.random.default_rng(2).standard_normal((5, E)).astype(np.float32)
    lg[0, :] = np.nan                       # all NaN: the lowest indices
    lg[1, [0, 5]] = np.nan                  # NaN where the largest would be
    lg[1, 5] = np.nan
    lg[2, :] = -np.inf
    lg[2, [3, 7]] = np.nan                  # NaN and -inf tie
    lg[3, 4] = np.inf
    lg[3, 2] = np.nan
    for k in (1, 4, E):
        idx, _ = orc.topk(lg, k)
        assert np.all((idx >= 0) & (idx < E))
        for t in range(lg.shape[0]):
            key = np.where(np.isnan(lg[t]), -np.inf, lg[t]).astype(np.float64)
            ref = np.lexsort((np.arange(E), -key))[:k]
            assert np.array_equal(idx[t], ref), (t, k)
    idx, _ = orc.topk(lg, 4)
    assert list(idx[0]) == [0, 1, 2, 3]
    assert list(idx[2]) == [0, 1, 2, 3]
    assert idx[3][0] == 4


def test_gates_closed_form(orc):
    rng = np.random.default_rng(7)
    T, E, k = 50, 16, 4
    lg = rng.standard_normal((T, E)).astype(np.float32) * 3
    idx, g0 = orc.topk(lg, k, renorm=0)
    idx1, g1 = orc.topk(lg, k, renorm=1)
    assert np.array_equal(idx, idx1)
    l64 = lg.astype(np.float64)
    p = np.exp(l64 - l64.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    ref0 = np.take_along_axis(p, idx.astype(np.int64), 1)
    assert np.max(np.abs(g0 - ref0)) <= 1e-6
    sel = np.take_along_axis(l64, idx.astype(np.int64), 1)
    q = np.exp(sel - sel.max(1, keepdims=True))
    ref1 = q / q.sum(1, keepdims=True)
    assert np.max(np.abs(g1 - ref1)) <= 1e-6
    assert np.max(np.abs(g1.sum(1) - 1)) <= 1e-6
    # descending gates follow descending logits
    assert np.all(np.diff(g0, axis=1) <= 0)
    # k = E with renorm = 1 is the full softmax
    _, gf = orc.topk(lg, E, renorm=1)
    _, gz = orc.topk(lg, E, renorm=0)
    assert np.max(np.abs(gf - gz)) <= 1e-7
    # one expert: gate is exactly 1
    _, g = orc.topk(lg[:, :1].copy(), 1, renorm=0)
    assert np.all(g == 1.0)


# ----------------------------------------------------------- permutation
@pytest.mark.parametrize("e_begin,E_loc", [(0, 12), (0, 5), (4, 3), (11, 1)])
def test_permutation_is_stable_argsort(orc, e_begin, E_loc):
    rng = np.random.default_rng(11)
    T, E, k = 200, 12, 3
    idx = np.stack([rng.choice(E, k, replace=False) for _ in range(T)]).astype(np.int32)
    pm = orc.permute_index(idx, E, e_begin, E_loc)
    flat = idx.ravel()
    assert np.array_equal(pm["counts_global"], np.bincount(flat, minlength=E))
    assert pm["counts_global"].sum() == T * k
    loc = (flat >= e_begin) & (flat < e_begin + E_loc)
    cnt = np.bincount(flat[loc] - e_begin, minlength=E_loc)
    assert np.array_equal(np.diff(pm["offsets"]), cnt)
    assert pm["offsets"][0] == 0 and pm["M"] == loc.sum()
    assert np.all(cnt <= T)
    a_loc = np.nonzero(loc)[0]
    order = a_loc[np.argsort(flat[a_loc], kind="stable")]
    assert np.array_equal(pm["row_src"], order)
    dst = pm["dst"].ravel()
    assert np.all(dst[~loc] == -1)
    assert np.array_equal(dst[pm["row_src"]], np.arange(pm["M"]))


def test_permute_unpermute_identity(orc):
    c = small_case(T=80, d=48, E=6, k=3, seed=2)
    lg = orc.logits(c["x"], c["w_r"])
    idx, _ = orc.topk(lg, 3)
    pm = orc.permute_index(idx, 6, 0, 6)
    xp = orc.gather(c["x"], pm["row_src"], 3)
    dst = pm["dst"]
    for t in range(80):
        for i in range(3):
            assert np.array_equal(xp[dst[t, i]], c["x"][t])
    # unit-weight combine of x_perm = k * x (exact: few bf16 terms in fp32)
    back = orc.combine(bits_to_f64(xp).astype(np.float32), dst, None)
    assert np.array_equal(back, 3 * bits_to_f64(c["x"]).astype(np.float32))


def test_combine_k1_is_inverse_permutation(orc):
    rng = np.random.default_rng(4)
    T, d = 30, 10
    dst = rng.permutation(T).astype(np.int32).reshape(T, 1)
    y = rng.standard_normal((T, d)).astype(np.float32)
    out = orc.combine(y, dst, np.ones((T, 1), np.float32))
    assert np.array_equal(out, y[dst[:, 0]])


# ------------------------------------------------------------- expert FFN
def _silu(z):
    return z / (1 + np.exp(-z))


def test_single_expert_is_dense_swiglu(orc):
    """E = 1, k = 1: the layer is a dense SwiGLU MLP (gate = 1)."""
    c = small_case(T=40, d=24, E=1, k=1, f=20, seed=9)
    o = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], 1, prec="f64")
    X = bits_to_f64(c["x"])
    Wg, Wu, Wd = (bits_to_f64(w)[0] for w in (c["wg"], c["wu"], c["wd"]))
    ref = (_silu(X @ Wg) * (X @ Wu)) @ Wd
    assert np.allclose(o["y"], ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())
    assert np.all(o["topk_gate"] == 1.0)


def test_per_expert_dense_mlp(orc):
    c = small_case(T=90, d=16, E=5, k=2, f=12, seed=21)
    o = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], None, 2, prec="f64")
    X = bits_to_f64(c["x"])
    off = o["offsets"]
    for e in range(5):
        rows = X[o["row_src"][off[e]:off[e + 1]] // 2]
        Wg, Wu, Wd = (bits_to_f64(w)[e] for w in (c["wg"], c["wu"], c["wd"]))
        ref = (_silu(rows @ Wg) * (rows @ Wu)) @ Wd
        assert np.allclose(o["y_perm"][off[e]:off[e + 1]], ref, rtol=1e-12, atol=1e-13)
    # combine closed form
    ref_y = np.zeros_like(o["y"])
    for t in range(90):
        for i in range(2):
            ref_y[t] += o["topk_gate"][t, i] * o["y_perm"][o["dst"][t, i]]
    assert np.allclose(o["y"], ref_y, rtol=1e-13, atol=1e-15)


# ---------------------------------------------------------- finite differences
def _fd_case(seed=0, T=5, d=8, E=4, k=2, f=6, renorm=0):
    rng = np.random.default_rng(seed)
    return dict(x=rng.standard_normal((T, d)), w_r=rng.standard_normal((d, E)),
                bias=rng.standard_normal(E) * 0.1,
                wg=rng.standard_normal((E, d, f)) * 0.5, wu=rng.standard_normal((E, d, f)) * 0.5,
                wd=rng.standard_normal((E, f, d)) * 0.5, dy=rng.standard_normal((T, d)),
                k=k, renorm=renorm)


def _loss(orc, c, **over):
    p = dict(c)
    p.update(over)
    o = orc.layer(p["x"], p["w_r"], p["bias"], p["wg"], p["wu"], p["wd"], None, p["k"],
                  renorm=p["renorm"], prec="f64_f64")
    return float(np.sum(o["y"] * c["dy"])), o["topk_idx"]


def _fd_check(orc, c, name, grad, h=1e-6, n=12, seed=0):
    rng = np.random.default_rng(seed)
    base = c[name]
    flat_idx = rng.choice(base.size, size=min(n, base.size), replace=False)
    _, idx0 = _loss(orc, c)
    for fi in flat_idx:
        pl = base.copy().ravel(); pl[fi] += h
        mi = base.copy().ravel(); mi[fi] -= h
        lp, ip = _loss(orc, c, **{name: pl.reshape(base.shape)})
        lm, im = _loss(orc, c, **{name: mi.reshape(base.shape)})
        assert np.array_equal(ip, idx0) and np.array_equal(im, idx0), "routing moved"
        fd = (lp - lm) / (2 * h)
        g = grad.ravel()[fi]
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(fd)), (name, fi, fd, g)


@pytest.mark.parametrize("renorm", [0, 1])
def test_layer_gradients_finite_differences(orc, renorm):
    c = _fd_case(seed=1 + renorm, renorm=renorm)
    o = orc.layer(c["x"], c["w_r"], c["bias"], c["wg"], c["wu"], c["wd"], c["dy"], c["k"],
                  renorm=renorm, prec="f64_f64", router_grad=True)
    _fd_check(orc, c, "wg", o["dw_gate"])
    _fd_check(orc, c, "wu", o["dw_up"])
    _fd_check(orc, c, "wd", o["dw_down"])
    _fd_check(orc, c, "w_r", o["dw_router"])
    _fd_check(orc, c, "bias", o["dbias"], n=4)
    _fd_check(orc, c, "x", o["dx_total"])


def test_gate_gradient_finite_differences(orc):
    """dgate = <dy_t, O_p>: perturb the gates directly in the combine."""
    c = _fd_case(seed=5)
    o = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], c["k"],
                  prec="f64_f64")
    h = 1e-6
    for t in range(c["x"].shape[0]):
        for i in range(c["k"]):
            gp = o["topk_gate"].copy(); gp[t, i] += h
            gm = o["topk_gate"].copy(); gm[t, i] -= h
            lp = np.sum(orc.combine(o["y_perm"], o["dst"], gp, "f64_f64") * c["dy"])
            lm = np.sum(orc.combine(o["y_perm"], o["dst"], gm, "f64_f64") * c["dy"])
            assert abs((lp - lm) / (2 * h) - o["dgate"][t, i]) <= 1e-7


def test_fp32_oracle_agrees_with_fp64(orc):
    c = small_case(T=128, d=64, E=8, k=2, f=96, seed=13)
    a = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], 2, prec="f32")
    b = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], 2, prec="f64")
    assert np.array_equal(a["topk_idx"], b["topk_idx"])
    for key in ("y", "dgate", "dx_perm", "dx", "dw_gate", "dw_up", "dw_down"):
        err = np.max(np.abs(a[key].astype(np.float64) - b[key]))
        assert err <= 1e-5 * np.max(np.abs(b[key])), key


# ----------------------------------------------------------- identities
def test_backward_bilinear_identities(orc):
    c = small_case(T=160, d=40, E=6, k=3, f=28, seed=17)
    o = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], 3, prec="f64")
    dy = bits_to_f64(c["dy"])
    # sum_i g_i dg_i = <dy_t, y_t>
    lhs = np.sum(o["topk_gate"] * o["dgate"], axis=1)
    rhs = np.sum(dy * o["y"], axis=1)
    assert np.allclose(lhs, rhs, rtol=1e-10, atol=1e-12)
    off = o["offsets"]
    X = bits_to_f64(o["x_perm"])
    for e in range(6):
        s = slice(off[e], off[e + 1])
        Wg, Wu, Wd = (bits_to_f64(w)[e] for w in (c["wg"], c["wu"], c["wd"]))
        tol = dict(rtol=1e-9, atol=1e-11)
        assert np.allclose(np.sum(o["dw_down"][e] * Wd), np.sum(o["dy_perm"][s] * o["y_perm"][s]), **tol)
        assert np.allclose(np.sum(o["dw_gate"][e] * Wg), np.sum(o["dh_gate"][s] * o["h_gate"][s]), **tol)
        assert np.allclose(np.sum(o["dw_up"][e] * Wu), np.sum(o["dh_up"][s] * o["h_up"][s]), **tol)
        assert np.allclose(np.sum(o["dx_perm"][s] * X[s]),
                           np.sum(o["dh_gate"][s] * o["h_gate"][s]) + np.sum(o["dh_up"][s] * o["h_up"][s]), **tol)


def test_empty_expert_has_exact_zero_gradients(orc):
    bias = np.zeros(6, np.float32)
    bias[[1, 4]] = -1.0e4
    c = small_case(T=70, d=16, E=6, k=2, f=8, seed=23, bias=bias)
    o = orc.layer(c["x"], c["w_r"], bias, c["wg"], c["wu"], c["wd"], c["dy"], 2, prec="f32")
    cnt = np.diff(o["offsets"])
    assert cnt[1] == 0 and cnt[4] == 0
    for e in (1, 4):
        assert np.all(o["dw_gate"][e] == 0) and np.all(o["dw_up"][e] == 0)
        assert np.all(o["dw_down"][e] == 0)
        assert not np.signbit(o["dw_gate"][e]).any()


def test_wgrad_entries_match_full(orc):
    c = small_case(T=100, d=24, E=3, k=2, f=16, seed=31)
    o = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], 2, prec="f64")
    off = o["offsets"]
    e = 1
    s = slice(off[e], off[e + 1])
    rng = np.random.default_rng(0)
    which = rng.integers(0, 3, 30)
    ii = np.where(which == 2, rng.integers(0, 16, 30), rng.integers(0, 24, 30))
    jj = np.where(which == 2, rng.integers(0, 24, 30), rng.integers(0, 16, 30))
    vals = orc.wgrad_entries(o["x_perm"][s], o["dy_perm"][s], c["wg"][e], c["wu"][e], c["wd"][e],
                             which, ii, jj, prec="f64")
    full = [o["dw_gate"][e], o["dw_up"][e], o["dw_down"][e]]
    ref = np.array([full[w][i, j] for w, i, j in zip(which, ii, jj)])
    assert np.allclose(vals, ref, rtol=1e-10, atol=1e-12)


def test_ep_share_filters_local_experts(orc):
    """Experts [e_begin, e_begin+E_loc) only: non-local slots give y = 0."""
    c = small_case(T=60, d=16, E=8, k=2, f=8, seed=41, E_loc=3, e_begin=2)
    o = orc.layer(c["x"], c["w_r"], None, c["wg"], c["wu"], c["wd"], c["dy"], 2,
                  e_begin=2, E_loc=3, prec="f32")
    loc = (o["topk_idx"] >= 2) & (o["topk_idx"] < 5)
    none = ~loc.any(1)
    assert none.any()
    assert np.all(o["y"][none] == 0) and np.all(o["dx"][none] == 0)
    assert np.all(o["dgate"][~loc] == 0)
    assert o["M"] == loc.sum()


def test_workload_generator_is_seeded():
    a = W.make_inputs("tiny", seed=0)
    b = W.make_inputs("tiny", seed=0)
    for key in ("x", "w_router", "w_gate", "w_up", "w_down", "dy"):
        assert np.array_equal(a[key].float().numpy(), b[key].float().numpy()), key
    wl = W.WORKLOADS["tiny"]
    assert a["x"].shape == (wl.T, wl.d) and a["w_down"].shape == (wl.E_loc, wl.f, wl.d)


def test_router_backward_entries_agree_with_full(orc):
    """The sampled router-backward helper (dot products in numpy) agrees with
    the full C routine (loops), which the finite-difference test pins."""
    rng = np.random.default_rng(7)
    T, d, E, k = 40, 24, 9, 3
    x = rng.normal(size=(T, d))
    w = 0.3 * rng.normal(size=(d, E))
    lg = x @ w
    idx, gate = orc.topk(lg, k, 0)
    dg = rng.normal(size=(T, k))
    for renorm in (0, 1):
        idx, gate = orc.topk(lg, k, renorm)
        dw, dx, db = orc.router_bwd_f64(x, w, lg, idx, gate, dg, renorm)
        dl = orc.router_dlogits_f64(lg, idx, gate, dg, renorm)
        jj, ee, tt = [0, 5, 23], [8, 0, 4], [0, 17, 39]
        dw_s, dx_s, db_s = orc.router_bwd_entries_f64(x, w, dl, jj, ee, tt)
        assert np.allclose(dw_s, dw[jj, ee], rtol=0, atol=1e-12)
        assert np.allclose(dx_s, dx[tt], rtol=0, atol=1e-12)
        assert np.allclose(db_s, db, rtol=0, atol=1e-12)
        # the logit gradients of one token sum to zero under renorm = 0 and 1
        # (softmax is invariant to a common shift of its logits)
        assert np.allclose(dl.sum(1), 0.0, atol=1e-12)
