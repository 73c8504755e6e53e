"""The C ABI without a GPU: the library loads, exports every function the
header declares, and rejects bad arguments on the host before any launch."""
import ctypes

import pytest

from paper_1907_13257_amd import lstm355 as L


@pytest.fixture(scope="module")
def lib():
    return L.load_library()


def test_exports_every_declared_symbol(lib):
    names = L.header_functions()
    assert {"lstm_create", "lstm_forward", "lstm_backward", "lstm_destroy"} <= set(names)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_status_strings(lib):
    for s, name in enumerate(["LSTM_OK", "LSTM_ERR_INVALID_ARG", "LSTM_ERR_UNSUPPORTED", "LSTM_ERR_WORKSPACE",
                              "LSTM_ERR_HIP", "LSTM_ERR_TIMEOUT"]):
        assert L.lstm_status_string(s) == name
    assert L.lstm_status_string(99) == "LSTM_ERR_UNKNOWN"


@pytest.mark.parametrize("kw", [
    dict(T=0), dict(B=0), dict(I=0), dict(H=-8), dict(Hp=-8),
    dict(I=12), dict(H=20), dict(Hp=4),
    dict(ldx=8), dict(ldx=36), dict(ldy=8),
])
def test_create_rejects_bad_descriptors(lib, kw):
    args = dict(T=4, B=3, I=32, H=16, Hp=0, dtype="bf16", reverse=False, ldx=0, ldy=0)
    args.update(kw)
    with pytest.raises(L.LSTMError) as e:
        L.lstm_create(**args)
    assert e.value.status == L.LSTM_ERR_INVALID_ARG


def test_create_rejects_bad_dtype_and_reverse(lib):
    h = ctypes.c_void_p()
    d = L.lstm_desc_t(4, 3, 32, 16, 0, 7, 0, 0, 0)
    assert lib.lstm_create(ctypes.byref(d), ctypes.byref(h)) == L.LSTM_ERR_INVALID_ARG
    d = L.lstm_desc_t(4, 3, 32, 16, 0, 1, 2, 0, 0)
    assert lib.lstm_create(ctypes.byref(d), ctypes.byref(h)) == L.LSTM_ERR_INVALID_ARG
    assert lib.lstm_create(None, ctypes.byref(h)) == L.LSTM_ERR_INVALID_ARG


def test_sizes_and_destroy(lib):
    T, B, I, H = 5, 3, 16, 24
    h = L.lstm_create(T, B, I, H, 0, "bf16")
    # reserve holds fp32 gates [T][B][4H] and cells [T][B][H]
    assert L.lstm_reserve_size(h) >= T * B * 4 * H * 4 + T * B * H * 4
    # workspace holds at least the bf16 gate gradients [T][B][4H]
    assert L.lstm_workspace_size(h) >= T * B * 4 * H * 2
    hp = L.lstm_create(T, B, I, H, 8, "f32")
    assert L.lstm_reserve_size(hp) >= T * B * 4 * H * 4 + T * B * H * 4 + T * B * H * 4
    L.lstm_destroy(h)
    L.lstm_destroy(hp)
    assert lib.lstm_destroy(None) == L.LSTM_OK
    assert lib.lstm_reserve_size(None) == 0


def test_forward_backward_validate_before_launch(lib):
    h = L.lstm_create(4, 3, 32, 16, 0, "bf16")
    A = 1 << 20  # a 16-byte aligned stand-in address; validation fails before any use
    R, WS = L.lstm_reserve_size(h), L.lstm_workspace_size(h)

    def fwd(hh, x=A, P=None, rb=R, wb=WS):
        return lib.lstm_forward(hh, x, None, None, A, A, A, P, A, None, None, A, rb, A, wb, None)

    # missing required pointers
    assert fwd(h, x=None) == L.LSTM_ERR_INVALID_ARG
    # P given to a plain LSTM
    assert fwd(h, P=A) == L.LSTM_ERR_INVALID_ARG
    # misaligned activation pointer
    assert fwd(h, x=A + 2) == L.LSTM_ERR_INVALID_ARG
    assert "aligned" in L.lstm_last_error_detail()
    assert fwd(None) == L.LSTM_ERR_INVALID_ARG

    # backward: missing weight gradients, bad accumulate flag
    def bwd(hh, P=None, dW=A, dP=None, acc=0, rb=R, wb=WS):
        return lib.lstm_backward(hh, A, None, None, A, None, None, A, A, P, A, A, rb, None, None, None,
                                 dW, A, A, dP, acc, A, wb, None)

    assert bwd(h, dW=None) == L.LSTM_ERR_INVALID_ARG
    assert bwd(h, acc=2) == L.LSTM_ERR_INVALID_ARG
    hp = L.lstm_create(4, 3, 32, 16, 8, "bf16")
    Rp, WSp = L.lstm_reserve_size(hp), L.lstm_workspace_size(hp)
    assert bwd(hp, P=A, rb=Rp, wb=WSp) == L.LSTM_ERR_INVALID_ARG   # dP missing
    L.lstm_destroy(h)
    L.lstm_destroy(hp)


def test_short_buffers_are_rejected_before_launch(lib):
    """A reserve or workspace shorter than the query functions report is
    LSTM_ERR_WORKSPACE, decided on the host (no device is touched)."""
    A = 1 << 20
    for Hp in (0, 8):
        h = L.lstm_create(5, 3, 32, 16, Hp, "bf16")
        R, WS = L.lstm_reserve_size(h), L.lstm_workspace_size(h)
        P = A if Hp else None
        dP = A if Hp else None

        def fwd(rb, wb):
            return lib.lstm_forward(h, A, None, None, A, A, A, P, A, None, None, A, rb, A, wb, None)

        def bwd(rb, wb):
            return lib.lstm_backward(h, A, None, None, A, None, None, A, A, P, A, A, rb, None, None, None,
                                     A, A, A, dP, 0, A, wb, None)

        for call in (fwd, bwd):
            assert call(R - 1, WS) == L.LSTM_ERR_WORKSPACE
            assert "reserve" in L.lstm_last_error_detail() and str(R) in L.lstm_last_error_detail()
            assert call(R, WS - 256) == L.LSTM_ERR_WORKSPACE
            assert "workspace" in L.lstm_last_error_detail()
            assert call(0, 0) == L.LSTM_ERR_WORKSPACE
        L.lstm_destroy(h)


def test_forward_stack_validates_before_launch(lib):
    """lstm_forward_stack rejects bad arguments and stacks the layer
    wavefront does not cover before anything touches the GPU."""
    import ctypes
    A = 1 << 20
    hb = [L.lstm_create(4, 8, 1024, 1024, 0, "bf16") for _ in range(5)]
    hf = [L.lstm_create(4, 8, 1024, 1024, 0, "f32") for _ in range(2)]
    arr = lambda vals: (ctypes.c_void_p * len(vals))(*vals)
    ptrs = lambda n: arr([A] * n)

    BIG = 1 << 60

    def call(hs, x=A, n=None, rb=BIG, wb=BIG):
        n = len(hs) if n is None else n
        return lib.lstm_forward_stack(n, arr(hs), x, ptrs(n), ptrs(n), ptrs(n), ptrs(n), None, None, ptrs(n), rb, A, wb,
                                      None)

    assert call(hb[:2], x=None) == L.LSTM_ERR_INVALID_ARG                  # missing input
    assert call(hb[:2], x=A + 2) == L.LSTM_ERR_INVALID_ARG                 # misaligned input
    assert call(hb[:2], n=0) == L.LSTM_ERR_INVALID_ARG
    assert call([hb[0], None]) == L.LSTM_ERR_INVALID_ARG                  # missing handle
    need_r, need_w = L.lstm_reserve_size(hb[0]), L.lstm_workspace_size(hb[0])
    assert call(hb[:2], rb=need_r - 1) == L.LSTM_ERR_WORKSPACE             # short reserves
    assert call(hb[:2], wb=need_w - 1) == L.LSTM_ERR_WORKSPACE             # short workspace
    assert call(hb[:1]) == L.LSTM_ERR_UNSUPPORTED                          # one layer
    assert call(hb[:5]) == L.LSTM_ERR_UNSUPPORTED                          # five layers
    assert call(hf) == L.LSTM_ERR_UNSUPPORTED                              # fp32
    assert "wavefront" in L.lstm_last_error_detail()
    # residual layers: a flag without its sum buffer, or on a layer whose input is narrower
    flags = (ctypes.c_int * 2)(0, 1)
    none2 = arr([None, None])
    assert lib.lstm_forward_stack(2, arr(hb[:2]), A, ptrs(2), ptrs(2), ptrs(2), ptrs(2), flags, none2, ptrs(2),
                                  BIG, A, BIG, None) == L.LSTM_ERR_INVALID_ARG
    assert "sum" in L.lstm_last_error_detail()
    hn = L.lstm_create(4, 8, 512, 1024, 0, "bf16")
    flags0 = (ctypes.c_int * 2)(1, 0)
    assert lib.lstm_forward_stack(2, arr([hn, hb[0]]), A, ptrs(2), ptrs(2), ptrs(2), ptrs(2), flags0, ptrs(2),
                                  ptrs(2), BIG, A, BIG, None) == L.LSTM_ERR_INVALID_ARG
    assert "wide" in L.lstm_last_error_detail()
    L.lstm_destroy(hn)
    hr = L.lstm_create(4, 8, 1024, 1024, 0, "bf16", reverse=True)
    assert call([hb[0], hr]) == L.LSTM_ERR_UNSUPPORTED                     # a reversed layer
    hw = L.lstm_create(4, 8, 512, 1024, 0, "bf16")
    assert call([hb[0], hw]) == L.LSTM_ERR_UNSUPPORTED                     # layer 1 input is not layer 0's y
    for h in hb + hf + [hr, hw]:
        L.lstm_destroy(h)


def test_backward_stack_validates_before_launch(lib):
    import ctypes
    A = 1 << 20
    arr = lambda vals: (ctypes.c_void_p * len(vals))(*vals)
    hb = [L.lstm_create(6, 8, 1024, 1024, 0, "bf16") for _ in range(3)]
    size = L.lstm_backward_stack_workspace_size(hb)
    tb = 6 * 8
    # per layer dz, below the top layer the gradient passed down; the kernels
    # read R and W themselves, so no transposed weights are kept
    assert 3 * tb * 4096 * 2 + 2 * tb * 1024 * 2 <= size < 3 * 4 * 1024 * 1024 * 2
    assert L.lstm_backward_stack_workspace_size(hb[:1]) == 0          # one layer
    h1 = L.lstm_create(1, 8, 1024, 1024, 0, "bf16")
    assert L.lstm_backward_stack_workspace_size([h1, h1]) == 0         # T = 1
    hn = L.lstm_create(6, 8, 512, 1024, 0, "bf16")
    assert L.lstm_backward_stack_workspace_size([hn, hb[0]]) == 0      # layer 0 input narrower than H

    BIG = 1 << 60

    def call(hs, dy=A, acc=0, rb=BIG, wb=BIG):
        n = len(hs)
        p = arr([A] * n)
        return lib.lstm_backward_stack(n, arr(hs), dy, A, p, p, p, None, None, p, rb, None, p, p, p, acc, A, wb, None)

    assert call(hb, dy=None) == L.LSTM_ERR_INVALID_ARG
    assert call(hb, acc=2) == L.LSTM_ERR_INVALID_ARG
    assert call(hb, dy=A + 2) == L.LSTM_ERR_INVALID_ARG
    assert call([hn, hb[0]]) == L.LSTM_ERR_UNSUPPORTED
    assert call([h1, h1]) == L.LSTM_ERR_UNSUPPORTED
    flags = (ctypes.c_int * 3)(1, 0, 0)   # the first layer's sum feeds the second layer's weight gradients
    p3 = arr([A] * 3)
    assert lib.lstm_backward_stack(3, arr(hb), A, A, p3, p3, p3, flags, arr([None] * 3), p3, BIG, None, p3, p3, p3,
                                   0, A, BIG, None) == L.LSTM_ERR_INVALID_ARG
    assert call(hb, rb=L.lstm_reserve_size(hb[0]) - 1) == L.LSTM_ERR_WORKSPACE
    assert call(hb, wb=size - 1) == L.LSTM_ERR_WORKSPACE
    assert "workspace" in L.lstm_last_error_detail()
    for h in hb + [h1, hn]:
        L.lstm_destroy(h)


def test_add_validates(lib):
    assert lib.lstm_add(5, 4, 1 << 20, 1 << 20, 1 << 20, None) == L.LSTM_ERR_INVALID_ARG
    assert lib.lstm_add(1, 4, None, 1 << 20, 1 << 20, None) == L.LSTM_ERR_INVALID_ARG
    assert lib.lstm_add(1, 0, None, None, None, None) == L.LSTM_OK


def test_profile_api_without_records(lib):
    L.lstm_profile_reset()
    assert L.lstm_profile_read() == {}


def test_noalloc_forward_validates_before_launch(lib):
    """lstm_forward_noalloc checks its arguments and the reserve's size on
    the host, like lstm_forward, before anything touches the GPU."""
    A = 1 << 20
    h = L.lstm_create(4, 3, 32, 16, 0, "bf16")
    R = L.lstm_reserve_size(h)

    def call(x=A, P=None, rb=R):
        return lib.lstm_forward_noalloc(h, x, None, None, A, A, A, P, A, None, None, A, rb, None)

    assert call(x=None) == L.LSTM_ERR_INVALID_ARG
    assert call(P=A) == L.LSTM_ERR_INVALID_ARG
    assert call(x=A + 2) == L.LSTM_ERR_INVALID_ARG
    assert call(rb=R - 1) == L.LSTM_ERR_WORKSPACE
    assert lib.lstm_forward_noalloc(None, A, None, None, A, A, A, None, A, None, None, A, R, None) \
        == L.LSTM_ERR_INVALID_ARG
    L.lstm_destroy(h)
