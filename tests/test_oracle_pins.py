"""Pins of the fp64 oracle against facts that do not come from the oracle
itself: central finite differences, closed forms of special cases, symmetry
and additivity properties of the LSTM recurrence, and an independent library
implementation (torch.nn.LSTM in float64 on the CPU, run as a black box).

Each pin is chosen so a plausible slip in the oracle (a swapped gate block, a
wrong sign, a dropped carry term, an off-by-one in the visiting order, a
transposed operand) makes at least one of them fail.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def normwise(a, r):
    a = np.asarray(a, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    den = np.max(np.abs(r)) if r.size else 0.0
    num = np.max(np.abs(a - r)) if r.size else 0.0
    return num / den if den > 0 else num


def rand_layer(rng, T, B, I, H, Hp=0, scale=0.5, state=True):
    Hr = Hp if Hp else H
    p = dict(
        x=rng.uniform(-1, 1, (T, B, I)),
        W=rng.uniform(-scale, scale, (4 * H, I)),
        R=rng.uniform(-scale, scale, (4 * H, Hr)),
        b=rng.uniform(-scale, scale, 4 * H),
        P=rng.uniform(-scale, scale, (Hp, H)) if Hp else None,
        h0=rng.uniform(-1, 1, (B, Hr)) if state else None,
        c0=rng.uniform(-1, 1, (B, H)) if state else None,
        dy=rng.standard_normal((T, B, Hr)),
        dhT=rng.standard_normal((B, Hr)),
        dcT=rng.standard_normal((B, H)),
    )
    return p


def layer_loss(p, reverse=False):
    o = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], p["P"], p["h0"], p["c0"], reverse=reverse)
    L = float(np.sum(p["dy"] * o["y"]))
    if p.get("dhT") is not None:
        L += float(np.sum(p["dhT"] * o["hT"]))
    if p.get("dcT") is not None:
        L += float(np.sum(p["dcT"] * o["cT"]))
    return L


def layer_grads(p, reverse=False):
    return oracle.layer_backward(p["x"], p["W"], p["R"], p["b"], p["dy"], p["P"], p["h0"], p["c0"],
                                 p.get("dhT"), p.get("dcT"), reverse=reverse)


def fd_check(p, key, gkey, grads, loss_fn, idx, tol=1e-6):
    """Central differences on the selected flat indices of p[key]."""
    arr = p[key]
    flat = arr.reshape(-1)
    got = grads[gkey].reshape(-1)[idx]
    ref = np.empty(len(idx))
    for n, i in enumerate(idx):
        v = flat[i]
        eps = 1e-6 * max(1.0, abs(v))
        flat[i] = v + eps
        lp = loss_fn(p)
        flat[i] = v - eps
        lm = loss_fn(p)
        flat[i] = v
        ref[n] = (lp - lm) / (2 * eps)
    err = normwise(got, ref)
    assert err <= tol, f"{gkey}: normwise FD error {err:.3e}"


def pick(rng, n, k):
    return np.arange(n) if n <= k else rng.choice(n, size=k, replace=False)


GRAD_KEYS = [("x", "dx"), ("h0", "dh0"), ("c0", "dc0"), ("b", "db"), ("W", "dW"), ("R", "dR")]


@pytest.mark.parametrize("reverse", [False, True])
def test_fd_tiny_lstm(reverse):
    """Every gradient of the 1-layer tiny LSTM (T=8, B=4, I=32, H=64)."""
    rng = np.random.default_rng(11 + reverse)
    p = rand_layer(rng, 8, 4, 32, 64, scale=1 / 8)
    g = layer_grads(p, reverse)
    fn = lambda q: layer_loss(q, reverse)
    for key, gk in GRAD_KEYS:
        fd_check(p, key, gk, g, fn, pick(rng, p[key].size, 256))


def test_fd_tiny_lstmp():
    """LSTMP gradients including dP (T=5, B=3, I=8, H=16, Hp=8)."""
    rng = np.random.default_rng(12)
    p = rand_layer(rng, 5, 3, 8, 16, Hp=8)
    g = layer_grads(p)
    for key, gk in GRAD_KEYS + [("P", "dP")]:
        fd_check(p, key, gk, g, layer_loss, np.arange(p[key].size))


def test_fd_tiny_lstmp_reverse():
    rng = np.random.default_rng(13)
    p = rand_layer(rng, 4, 2, 8, 12, Hp=4)
    g = layer_grads(p, True)
    fn = lambda q: layer_loss(q, True)
    for key, gk in GRAD_KEYS + [("P", "dP")]:
        fd_check(p, key, gk, g, fn, np.arange(p[key].size))


def _tiny_stack(rng, T=4, B=3, I=6, H=4):
    """Bidirectional layer 1 (I -> 2H), layer 2 (2H -> H), residual layer 3."""
    def prm(i, h, state=False):
        d = dict(W=rng.uniform(-0.5, 0.5, (4 * h, i)), R=rng.uniform(-0.5, 0.5, (4 * h, h)),
                 b=rng.uniform(-0.5, 0.5, 4 * h))
        if state:
            d["h0"] = rng.uniform(-1, 1, (B, h))
            d["c0"] = rng.uniform(-1, 1, (B, h))
        return d
    layers = [oracle.LayerDef([prm(I, H, True), prm(I, H, True)]),
              oracle.LayerDef([prm(2 * H, H)]),
              oracle.LayerDef([prm(H, H)], residual=True)]
    x = rng.uniform(-1, 1, (T, B, I))
    d_out = rng.standard_normal((T, B, H))
    return x, layers, d_out


def test_fd_stack_bidirectional_residual():
    rng = np.random.default_rng(14)
    x, layers, d_out = _tiny_stack(rng)
    g = oracle.stack_backward(x, layers, d_out)

    def loss():
        y, _ = oracle.stack_forward(x, layers)
        return float(np.sum(d_out * y))

    def fd(arr, got):
        flat = arr.reshape(-1)
        ref = np.empty(flat.size)
        for i in range(flat.size):
            v = flat[i]
            eps = 1e-6 * max(1.0, abs(v))
            flat[i] = v + eps
            lp = loss()
            flat[i] = v - eps
            lm = loss()
            flat[i] = v
            ref[i] = (lp - lm) / (2 * eps)
        assert normwise(got.reshape(-1), ref) <= 1e-6

    fd(x, g["dx"])
    for li, L in enumerate(layers):
        for d, prm in enumerate(L.dirs):
            gd = g["layers"][li][d]
            for key, gk in [("W", "dW"), ("R", "dR"), ("b", "db"), ("h0", "dh0"), ("c0", "dc0")]:
                if key in prm:
                    fd(prm[key], gd[gk])


def _sig(u):
    return 1.0 / (1.0 + math.exp(-u))


def test_closed_form_zero_weights():
    """W = R = 0: the cell follows c_t = s + a c_{t-1}, a = sig(b_f),
    s = sig(b_i) tanh(b_g), so c_t = a^t c_0 + s (1 - a^t) / (1 - a) and
    h_t = sig(b_o) tanh(c_t), whatever x and h0 are.  Backward: dx and dh0 are
    exactly zero, dc0 = sum_t dy_t sig(b_o) (1 - tanh^2 c_t) a^t."""
    rng = np.random.default_rng(15)
    T, B, I, H = 7, 3, 5, 4
    p = rand_layer(rng, T, B, I, H)
    p["W"][:] = 0
    p["R"][:] = 0
    p["dhT"] = None
    p["dcT"] = None
    b = p["b"]
    o = oracle.layer_forward(p["x"], p["W"], p["R"], b, None, p["h0"], p["c0"])
    g = layer_grads(p)
    for j in range(H):
        a = _sig(b[H + j])
        s = _sig(b[j]) * math.tanh(b[2 * H + j])
        so = _sig(b[3 * H + j])
        for bb in range(B):
            c0 = p["c0"][bb, j]
            dc0 = 0.0
            for t in range(T):
                n = t + 1
                c = a ** n * c0 + s * (1 - a ** n) / (1 - a)
                h = so * math.tanh(c)
                assert abs(o["y"][t, bb, j] - h) <= 1e-14
                dc0 += p["dy"][t, bb, j] * so * (1 - math.tanh(c) ** 2) * a ** n
            assert abs(o["cT"][bb, j] - c) <= 1e-14
            assert abs(g["dc0"][bb, j] - dc0) <= 1e-13 * max(1.0, abs(dc0))
    assert np.all(g["dx"] == 0.0)
    assert np.all(g["dh0"] == 0.0)
    # the output does not depend on x or h0
    o2 = oracle.layer_forward(p["x"] * 3 + 1, p["W"], p["R"], b, None, -p["h0"], p["c0"])
    assert np.array_equal(o["y"], o2["y"])


def test_scalar_hand_case():
    """T = B = I = H = 1, h0 = c0 = 0, x = 1, b = 0: z = W, so
    c_1 = sig(w_i) tanh(w_g) and h_1 = sig(w_o) tanh(c_1); R has no effect."""
    W = np.array([[0.3], [-0.7], [1.1], [0.45]])
    for R in (np.zeros((4, 1)), np.array([[2.0], [-3.0], [0.5], [1.5]])):
        o = oracle.layer_forward(np.ones((1, 1, 1)), W, R, np.zeros(4))
        c1 = _sig(0.3) * math.tanh(1.1)
        h1 = _sig(0.45) * math.tanh(c1)
        assert abs(o["cT"][0, 0] - c1) <= 1e-15
        assert abs(o["y"][0, 0, 0] - h1) <= 1e-15


def test_saturated_memory_path():
    """b_f >> 0, b_i << 0, W = R = 0: the cell keeps c_0 and
    dc0 ~= sum_t dy_t sig(b_o) (1 - tanh^2 c_0)."""
    T, B, H = 6, 2, 3
    rng = np.random.default_rng(16)
    b = np.zeros(4 * H)
    b[:H] = -40.0
    b[H:2 * H] = 40.0
    b[3 * H:] = rng.uniform(-1, 1, H)
    c0 = rng.uniform(-1, 1, (B, H))
    dy = rng.standard_normal((T, B, H))
    x = rng.uniform(-1, 1, (T, B, 2))
    Z2 = np.zeros((4 * H, 2))
    ZH = np.zeros((4 * H, H))
    o = oracle.layer_forward(x, Z2, ZH, b, None, None, c0)
    g = oracle.layer_backward(x, Z2, ZH, b, dy, None, None, c0)
    so = 1 / (1 + np.exp(-b[3 * H:]))
    assert np.allclose(o["cT"], c0, atol=1e-12)
    want = dy.sum(axis=0) * so * (1 - np.tanh(c0) ** 2)
    assert np.allclose(g["dc0"], want, atol=1e-12)


def test_lstmp_identity_projection_is_lstm():
    """Hp = H with P = I reduces LSTMP to the plain LSTM."""
    rng = np.random.default_rng(17)
    p = rand_layer(rng, 5, 3, 6, 8)
    eye = np.eye(8)
    a = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], None, p["h0"], p["c0"])
    bq = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], eye, p["h0"], p["c0"])
    for k in ("y", "hT", "cT"):
        assert normwise(bq[k], a[k]) <= 1e-15
    ga = layer_grads(p)
    q = dict(p, P=eye)
    gb = layer_grads(q)
    for k in ("dx", "dh0", "dc0", "dW", "dR", "db"):
        assert normwise(gb[k], ga[k]) <= 1e-14


@pytest.mark.parametrize("Hp", [0, 4])
def test_batch_permutation_equivariance(Hp):
    rng = np.random.default_rng(18)
    p = rand_layer(rng, 5, 6, 7, 8, Hp=Hp)
    perm = rng.permutation(6)
    q = dict(p)
    q["x"] = p["x"][:, perm]
    q["dy"] = p["dy"][:, perm]
    for k in ("h0", "c0", "dhT", "dcT"):
        q[k] = p[k][perm]
    a = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], p["P"], p["h0"], p["c0"])
    b = oracle.layer_forward(q["x"], q["W"], q["R"], q["b"], q["P"], q["h0"], q["c0"])
    assert np.array_equal(a["y"][:, perm], b["y"])
    assert np.array_equal(a["cT"][perm], b["cT"])
    ga, gb = layer_grads(p), layer_grads(q)
    assert np.array_equal(ga["dx"][:, perm], gb["dx"])
    assert np.array_equal(ga["dh0"][perm], gb["dh0"])
    assert np.array_equal(ga["dc0"][perm], gb["dc0"])
    for k in ("dW", "dR", "db") + (("dP",) if Hp else ()):
        assert normwise(gb[k], ga[k]) <= 1e-13


@pytest.mark.parametrize("Hp", [0, 4])
def test_batch_split_additivity(Hp):
    """dW(B1 u B2) = dW(B1) + dW(B2): the identity the data-parallel gradient
    all-reduce relies on."""
    rng = np.random.default_rng(19)
    p = rand_layer(rng, 4, 7, 5, 8, Hp=Hp)
    sel = [np.arange(3), np.arange(3, 7)]
    parts = []
    for s in sel:
        q = dict(p)
        q["x"] = p["x"][:, s]
        q["dy"] = p["dy"][:, s]
        for k in ("h0", "c0", "dhT", "dcT"):
            q[k] = p[k][s]
        parts.append(layer_grads(q))
    full = layer_grads(p)
    for k in ("dW", "dR", "db") + (("dP",) if Hp else ()):
        assert normwise(parts[0][k] + parts[1][k], full[k]) <= 1e-13


def test_hidden_unit_permutation():
    """Relabelling the cells (consistently in every gate block, in R's columns,
    h0, c0 and the gradients) relabels every result."""
    rng = np.random.default_rng(20)
    T, B, I, H = 4, 3, 5, 6
    p = rand_layer(rng, T, B, I, H)
    pi = rng.permutation(H)
    rows = np.concatenate([g * H + pi for g in range(4)])
    q = dict(p)
    q["W"] = p["W"][rows]
    q["R"] = p["R"][rows][:, pi]
    q["b"] = p["b"][rows]
    q["h0"] = p["h0"][:, pi]
    q["c0"] = p["c0"][:, pi]
    q["dy"] = p["dy"][:, :, pi]
    q["dhT"] = p["dhT"][:, pi]
    q["dcT"] = p["dcT"][:, pi]
    a = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], None, p["h0"], p["c0"])
    b = oracle.layer_forward(q["x"], q["W"], q["R"], q["b"], None, q["h0"], q["c0"])
    assert normwise(b["y"], a["y"][:, :, pi]) <= 1e-15
    ga, gb = layer_grads(p), layer_grads(q)
    assert normwise(gb["dx"], ga["dx"]) <= 1e-14
    assert normwise(gb["dW"], ga["dW"][rows]) <= 1e-14
    assert normwise(gb["dR"], ga["dR"][rows][:, pi]) <= 1e-14
    assert normwise(gb["dh0"], ga["dh0"][:, pi]) <= 1e-14


@pytest.mark.parametrize("Hp", [0, 3])
def test_time_reversal(Hp):
    """reverse=1 on x equals the forward direction on x flipped in time,
    flipped back; gradients likewise."""
    rng = np.random.default_rng(21)
    p = rand_layer(rng, 6, 2, 4, 5, Hp=Hp)
    q = dict(p)
    q["x"] = p["x"][::-1].copy()
    q["dy"] = p["dy"][::-1].copy()
    a = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], p["P"], p["h0"], p["c0"], reverse=True)
    b = oracle.layer_forward(q["x"], q["W"], q["R"], q["b"], q["P"], q["h0"], q["c0"])
    assert np.array_equal(a["y"], b["y"][::-1])
    assert np.array_equal(a["hT"], b["hT"])
    ga, gb = layer_grads(p, True), layer_grads(q, False)
    assert np.array_equal(ga["dx"], gb["dx"][::-1])
    for k in ("dW", "dR", "db", "dh0", "dc0"):
        assert normwise(ga[k], gb[k]) <= 1e-14


@pytest.mark.parametrize("Hp", [0, 4])
def test_state_carry(Hp):
    """Forward over T1 + T2 steps equals T1 steps, then T2 steps started from
    (hT, cT); backward chains through dhT / dcT the same way."""
    rng = np.random.default_rng(22)
    T1, T2 = 3, 4
    p = rand_layer(rng, T1 + T2, 3, 5, 6, Hp=Hp)
    full = oracle.layer_forward(p["x"], p["W"], p["R"], p["b"], p["P"], p["h0"], p["c0"])
    a = oracle.layer_forward(p["x"][:T1], p["W"], p["R"], p["b"], p["P"], p["h0"], p["c0"])
    b = oracle.layer_forward(p["x"][T1:], p["W"], p["R"], p["b"], p["P"], a["hT"], a["cT"])
    assert normwise(np.concatenate([a["y"], b["y"]]), full["y"]) <= 1e-15
    assert normwise(b["cT"], full["cT"]) <= 1e-15
    gfull = layer_grads(p)
    g2 = oracle.layer_backward(p["x"][T1:], p["W"], p["R"], p["b"], p["dy"][T1:], p["P"], a["hT"], a["cT"],
                               p["dhT"], p["dcT"])
    g1 = oracle.layer_backward(p["x"][:T1], p["W"], p["R"], p["b"], p["dy"][:T1], p["P"], p["h0"], p["c0"],
                               g2["dh0"], g2["dc0"])
    assert normwise(np.concatenate([g1["dx"], g2["dx"]]), gfull["dx"]) <= 1e-14
    assert normwise(g1["dh0"], gfull["dh0"]) <= 1e-14
    assert normwise(g1["dc0"], gfull["dc0"]) <= 1e-14
    for k in ("dW", "dR", "db") + (("dP",) if Hp else ()):
        assert normwise(g1[k] + g2[k], gfull[k]) <= 1e-13


def test_backward_linearity():
    rng = np.random.default_rng(23)
    p = rand_layer(rng, 5, 3, 4, 6, Hp=3)
    q = dict(p)
    q["dy"] = rng.standard_normal(p["dy"].shape)
    q["dhT"] = rng.standard_normal(p["dhT"].shape)
    q["dcT"] = rng.standard_normal(p["dcT"].shape)
    al, be = 0.7, -1.9
    r = dict(p)
    for k in ("dy", "dhT", "dcT"):
        r[k] = al * p[k] + be * q[k]
    gp, gq, gr = layer_grads(p), layer_grads(q), layer_grads(r)
    for k in gp:
        assert normwise(gr[k], al * gp[k] + be * gq[k]) <= 1e-13


# ---------------------------------------------------------------------------
# independent library implementation
# ---------------------------------------------------------------------------
torch = pytest.importorskip("torch")


def _torch_run(p, Hp, bidir, rev_p=None):
    T, B, I = p["x"].shape
    H = p["W"].shape[0] // 4
    Hr = Hp if Hp else H
    D = 2 if bidir else 1
    m = torch.nn.LSTM(I, H, proj_size=Hp, bidirectional=bidir, dtype=torch.float64)
    sets = [("", p)] + ([("_reverse", rev_p)] if bidir else [])
    with torch.no_grad():
        for sfx, q in sets:
            getattr(m, "weight_ih_l0" + sfx).copy_(torch.from_numpy(q["W"]))
            getattr(m, "weight_hh_l0" + sfx).copy_(torch.from_numpy(q["R"]))
            getattr(m, "bias_ih_l0" + sfx).copy_(torch.from_numpy(q["b"]))
            getattr(m, "bias_hh_l0" + sfx).zero_()
            if Hp:
                getattr(m, "weight_hr_l0" + sfx).copy_(torch.from_numpy(q["P"]))
    x = torch.from_numpy(p["x"]).requires_grad_(True)
    h0 = torch.from_numpy(np.stack([q["h0"] for _, q in sets])).requires_grad_(True)
    c0 = torch.from_numpy(np.stack([q["c0"] for _, q in sets])).requires_grad_(True)
    y, (hn, cn) = m(x, (h0, c0))
    dy = np.concatenate([q["dy"] for _, q in sets], axis=2)
    L = (y * torch.from_numpy(dy)).sum()
    L = L + (hn * torch.from_numpy(np.stack([q["dhT"] for _, q in sets]))).sum()
    L = L + (cn * torch.from_numpy(np.stack([q["dcT"] for _, q in sets]))).sum()
    L.backward()
    out = []
    for d, (sfx, q) in enumerate(sets):
        g = dict(y=y.detach().numpy()[:, :, d * Hr:(d + 1) * Hr], hT=hn.detach().numpy()[d],
                 cT=cn.detach().numpy()[d], dh0=h0.grad.numpy()[d], dc0=c0.grad.numpy()[d],
                 dW=getattr(m, "weight_ih_l0" + sfx).grad.numpy(),
                 dR=getattr(m, "weight_hh_l0" + sfx).grad.numpy(),
                 db=getattr(m, "bias_ih_l0" + sfx).grad.numpy())
        if Hp:
            g["dP"] = getattr(m, "weight_hr_l0" + sfx).grad.numpy()
        out.append(g)
    return out, x.grad.numpy()


@pytest.mark.parametrize("Hp", [0, 5])
@pytest.mark.parametrize("bidir", [False, True])
def test_torch_lstm_cross_check(Hp, bidir):
    rng = np.random.default_rng(24)
    T, B, I, H = 6, 3, 7, 9
    p = rand_layer(rng, T, B, I, H, Hp=Hp)
    q = rand_layer(rng, T, B, I, H, Hp=Hp)
    q["x"] = p["x"]
    ref, dx_ref = _torch_run(p, Hp, bidir, q if bidir else None)
    dx = 0
    for d, prm in enumerate([p, q] if bidir else [p]):
        o = oracle.layer_forward(prm["x"], prm["W"], prm["R"], prm["b"], prm["P"], prm["h0"], prm["c0"],
                                 reverse=(d == 1))
        g = layer_grads(prm, reverse=(d == 1))
        for k in ("y", "hT", "cT"):
            assert normwise(o[k], ref[d][k]) <= 1e-12, k
        for k in ("dh0", "dc0", "dW", "dR", "db") + (("dP",) if Hp else ()):
            assert normwise(g[k], ref[d][k]) <= 1e-12, k
        dx = dx + g["dx"]
    assert normwise(dx, dx_ref) <= 1e-12


# ---------------------------------------------------------------------------
# stored regression values
# ---------------------------------------------------------------------------
def test_golden_regression():
    """Values written by tests/golden/make_golden.py (which calls only the
    oracle) for a small hand-specified layer; catches silent changes."""
    with open(os.path.join(GOLDEN, "small_layer.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        inp = {k: (None if v is None else np.array(v, dtype=np.float64)) for k, v in case["inputs"].items()}
        o = oracle.layer_forward(inp["x"], inp["W"], inp["R"], inp["b"], inp["P"], inp["h0"], inp["c0"],
                                 reverse=case["reverse"])
        g = oracle.layer_backward(inp["x"], inp["W"], inp["R"], inp["b"], inp["dy"], inp["P"], inp["h0"],
                                  inp["c0"], inp["dhT"], inp["dcT"], reverse=case["reverse"])
        res = dict(o, **g)
        for k, v in case["expected"].items():
            assert normwise(res[k], np.array(v)) <= 1e-14, (case["name"], k)


def test_torch_stack_cross_check():
    """Stack composition against torch in float64 on the CPU, run as a black
    box: torch.nn.LSTM(num_layers=2, bidirectional=True) for a bidirectional
    first layer whose concatenated output feeds a bidirectional second layer,
    then a unidirectional third layer with its residual added by hand.  The
    oracle composes the same three layers with stack_forward / stack_backward
    (concatenation order, split of the upstream gradient between directions,
    summed input gradients, identity path of the residual)."""
    rng = np.random.default_rng(31)
    T, B, I, H = 5, 3, 6, 4
    W = lambda *s: rng.uniform(-0.6, 0.6, s)
    p = [[dict(W=W(4 * H, I), R=W(4 * H, H), b=W(4 * H)) for _ in range(2)],
         [dict(W=W(4 * H, 2 * H), R=W(4 * H, H), b=W(4 * H)) for _ in range(2)],
         [dict(W=W(4 * (2 * H), 2 * H), R=W(4 * (2 * H), 2 * H), b=W(4 * (2 * H)))]]
    # the third layer has 2H cells so that its residual (output = y + input) is defined
    x = rng.uniform(-1, 1, (T, B, I))
    dy = rng.standard_normal((T, B, 2 * H))

    m = torch.nn.LSTM(I, H, num_layers=2, bidirectional=True, dtype=torch.float64)
    m3 = torch.nn.LSTM(2 * H, 2 * H, dtype=torch.float64)
    with torch.no_grad():
        for l in range(2):
            for d, sfx in enumerate(("", "_reverse")):
                getattr(m, f"weight_ih_l{l}{sfx}").copy_(torch.from_numpy(p[l][d]["W"]))
                getattr(m, f"weight_hh_l{l}{sfx}").copy_(torch.from_numpy(p[l][d]["R"]))
                getattr(m, f"bias_ih_l{l}{sfx}").copy_(torch.from_numpy(p[l][d]["b"]))
                getattr(m, f"bias_hh_l{l}{sfx}").zero_()
        m3.weight_ih_l0.copy_(torch.from_numpy(p[2][0]["W"]))
        m3.weight_hh_l0.copy_(torch.from_numpy(p[2][0]["R"]))
        m3.bias_ih_l0.copy_(torch.from_numpy(p[2][0]["b"]))
        m3.bias_hh_l0.zero_()
    xt = torch.from_numpy(x).requires_grad_(True)
    y2, _ = m(xt)
    y3, _ = m3(y2)
    out = y3 + y2
    (out * torch.from_numpy(dy)).sum().backward()

    layers = [oracle.LayerDef(p[0]), oracle.LayerDef(p[1]), oracle.LayerDef(p[2], residual=True)]
    o, _ = oracle.stack_forward(x, layers)
    g = oracle.stack_backward(x, layers, dy)
    assert normwise(o, out.detach().numpy()) <= 1e-12
    assert normwise(g["dx"], xt.grad.numpy()) <= 1e-12
    for l in range(2):
        for d, sfx in enumerate(("", "_reverse")):
            assert normwise(g["layers"][l][d]["dW"], getattr(m, f"weight_ih_l{l}{sfx}").grad.numpy()) <= 1e-12
            assert normwise(g["layers"][l][d]["dR"], getattr(m, f"weight_hh_l{l}{sfx}").grad.numpy()) <= 1e-12
            assert normwise(g["layers"][l][d]["db"], getattr(m, f"bias_ih_l{l}{sfx}").grad.numpy()) <= 1e-12
    assert normwise(g["layers"][2][0]["dW"], m3.weight_ih_l0.grad.numpy()) <= 1e-12
    assert normwise(g["layers"][2][0]["dR"], m3.weight_hh_l0.grad.numpy()) <= 1e-12
    assert normwise(g["layers"][2][0]["db"], m3.bias_ih_l0.grad.numpy()) <= 1e-12
