"""The allocation-free conv entry point against ctc_conv2d_forward.

ctc_conv2d_forward_noalloc keeps the fp32 partial sums of split-K layers in
the library's static scratch array instead of a caller workspace.  Two calls
in a row on one GPU (the second with fewer images, so it leaves part of the
first call's partial sums in the array) must give exactly the outputs of
ctc_conv2d_forward with a workspace, which takes the same kernels and the
same k ranges; a layer whose partial sums exceed the array is refused
before anything runs.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctc():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_16742_amd import ctc
    return ctc


def _pack_krsc(w):
    return np.ascontiguousarray(w.transpose(0, 2, 3, 1))


def _run_pair(ctc, dt, n, C, H, K, seed):
    tdt = torch.float16 if dt == "f16" else torch.float32
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, H, H, C)).astype(np.float32)
    w = (rng.standard_normal((K, C, 3, 3)) / np.sqrt(9 * C)).astype(np.float32)
    d = ctc.layer_desc(C, K, 3, 3, 1, 1, 1, 0, ctc.CTC_ROLE_NONE)
    xd = torch.from_numpy(x).to("cuda", tdt)
    wd = torch.from_numpy(_pack_krsc(w)).to("cuda", tdt)
    sd = torch.from_numpy(rng.uniform(0.5, 1.5, K).astype(np.float32)).cuda()
    hd = torch.from_numpy(rng.standard_normal(K).astype(np.float32)).cuda()
    nb = ctc.ctc_conv2d_workspace_bytes(d, ctc.DTYPES[dt], n, H, H)
    ws = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda")
    y_ws = torch.full((n, H, H, K), float("nan"), dtype=tdt, device="cuda")
    y_na = torch.full_like(y_ws, float("nan"))
    ctc.ctc_conv2d_forward(d, ctc.DTYPES[dt], n, H, H, xd, wd, sd, hd, None, 1,
                           y_ws, workspace=ws, ws_bytes=nb)
    ctc.ctc_conv2d_forward_noalloc(d, ctc.DTYPES[dt], n, H, H, xd, wd, sd, hd,
                                   None, 1, y_na)
    torch.cuda.synchronize()
    a = y_ws.cpu().numpy()
    b = y_na.cpu().numpy()
    assert not np.isnan(a).any()
    view = np.uint16 if dt == "f16" else np.uint32
    assert np.array_equal(a.view(view), b.view(view))
    return nb


@pytest.mark.parametrize("dt", ["f16", "f32"])
def test_noalloc_conv_equals_workspace_conv_twice(ctc, dt):
    """K = 4608 on 8x8 maps (four k ranges): 8 images, then 3, each
    bit-identical to the workspace call."""
    nb8 = _run_pair(ctc, dt, 8, 512, 8, 512, 1)
    nb3 = _run_pair(ctc, dt, 3, 512, 8, 512, 2)
    assert nb8 == 4 * 8 * 64 * 512 * 4 and nb3 < nb8


def test_noalloc_conv_without_split(ctc):
    """A layer that does not split K runs the same kernel either way."""
    assert _run_pair(ctc, "f16", 2, 64, 20, 128, 3) == 0


def test_noalloc_conv_rejects_partial_sums_beyond_the_scratch(ctc):
    """128 images of the 8x8 x 512 layer need 67 MB of partial sums: refused
    with CTC_ERR_WORKSPACE, output untouched."""
    d = ctc.layer_desc(512, 512, 3, 3, 1, 1, 1, 0, ctc.CTC_ROLE_NONE)
    n = 128
    assert ctc.ctc_conv2d_workspace_bytes(d, ctc.CTC_F16, n, 8, 8) > 32 << 20
    x = torch.zeros((n, 8, 8, 512), dtype=torch.float16, device="cuda")
    w = torch.zeros((512, 3, 3, 512), dtype=torch.float16, device="cuda")
    s = torch.ones(512, device="cuda")
    y = torch.full_like(x, 7.0)
    with pytest.raises(ctc.CtcError) as e:
        ctc.ctc_conv2d_forward_noalloc(d, ctc.CTC_F16, n, 8, 8, x, w, s, s,
                                       None, 1, y)
    assert e.value.status == ctc.CTC_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
