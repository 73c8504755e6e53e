"""lstm_forward_noalloc (the forward pass with the library's own device
scratch instead of a workspace argument) against lstm_forward, through the
C ABI: two calls in a row on one GPU, the second with a smaller layer, each
bitwise equal to lstm_forward on the same inputs (same kernels, same order of
arithmetic) and within the bf16 / fp32 tolerance of the oracle."""
import numpy as np
import pytest

from _gpu_helpers import TOL, announce, normwise, to_dev, to_f64
from test_gpu_parity import layer_case, oracle_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def forward_both(T, B, I, H, dtype, seed):
    from paper_1907_13257_amd import lstm355 as L
    c = layer_case(T, B, I, H, 0, dtype, False, seed=seed)
    d = {k: to_dev(v) for k, v in c.items()}
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    h = L.lstm_create(T, B, I, H, 0, dtype)
    res = {}
    try:
        for mode in ("workspace", "noalloc"):
            y = torch.full((T, B, H), float("nan"), dtype=td, device="cuda")
            hT = torch.full((B, H), float("nan"), dtype=td, device="cuda")
            cT = torch.full((B, H), float("nan"), dtype=torch.float32, device="cuda")
            reserve = torch.empty(L.lstm_reserve_size(h), dtype=torch.uint8, device="cuda")
            if mode == "workspace":
                ws = torch.empty(L.lstm_workspace_size(h), dtype=torch.uint8, device="cuda")
                L.lstm_forward(h, d["x"], d["h0"], d["c0"], d["W"], d["R"], d["b"], None, y, hT, cT, reserve, ws)
            else:
                L.lstm_forward_noalloc(h, d["x"], d["h0"], d["c0"], d["W"], d["R"], d["b"], None, y, hT, cT,
                                       reserve)
            assert L.lstm_check(h, None) == L.LSTM_OK
            torch.cuda.synchronize()
            res[mode] = dict(y=to_f64(y), hT=to_f64(hT), cT=to_f64(cT))
    finally:
        L.lstm_destroy(h)
    return c, res


@pytest.mark.parametrize("dtype,first,second", [
    ("bf16", (6, 40, 64, 256), (3, 9, 32, 256)),     # XCD-local recurrence, then a smaller layer
    ("f32", (5, 37, 40, 72), (2, 5, 16, 40)),        # generic persistent recurrence (grid barrier)
])
def test_noalloc_forward_matches_workspace_forward(dtype, first, second):
    for i, (T, B, I, H) in enumerate((first, second)):
        label = f"noalloc call {i + 1}: T{T} B{B} I{I} H{H} {dtype}"
        announce(label)
        c, res = forward_both(T, B, I, H, dtype, seed=100 + 10 * i + T)
        for k in ("y", "hT", "cT"):
            assert np.array_equal(res["noalloc"][k], res["workspace"][k]), (label, k)
        ref = oracle_layer(c, 0, False)
        errs = {k: normwise(res["noalloc"][k], ref[k]) for k in ("y", "hT", "cT")}
        announce(f"{label} errors vs oracle: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
        assert max(errs.values()) <= TOL[dtype]["out"], errs


def test_noalloc_rejects_a_layer_needing_more_scratch():
    """The stepwise recurrence of a wide LSTMP layer needs split-K partials
    beyond the library's scratch: a clear LSTM_ERR_WORKSPACE, nothing launched."""
    from paper_1907_13257_amd import lstm355 as L
    T, B, I, H, Hp = 2, 8, 64, 2048, 256
    h = L.lstm_create(T, B, I, H, Hp, "bf16")
    try:
        z = lambda *s: torch.zeros(s, dtype=torch.bfloat16, device="cuda")
        x, W, R, P = z(T, B, I), z(4 * H, I), z(4 * H, Hp), z(Hp, H)
        b = torch.zeros(4 * H, dtype=torch.float32, device="cuda")
        y = z(T, B, Hp)
        reserve = torch.empty(L.lstm_reserve_size(h), dtype=torch.uint8, device="cuda")
        st = L.load_library().lstm_forward_noalloc(h, x.data_ptr(), None, None, W.data_ptr(), R.data_ptr(),
                                                   b.data_ptr(), P.data_ptr(), y.data_ptr(), None, None,
                                                   reserve.data_ptr(), reserve.numel(), None)
        assert st == L.LSTM_ERR_WORKSPACE
        assert "scratch" in L.lstm_last_error_detail()
    finally:
        L.lstm_destroy(h)
