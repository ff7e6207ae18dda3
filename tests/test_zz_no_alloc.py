"""The allocation-free weight gradient (rat3d_conv3d_wgrad_noalloc, scratch in
a library-owned device array) against rat3d_conv3d_wgrad with a caller
workspace, on two calls in a row per kernel family, the second with a smaller
input (the scratch keeps the first call's partials, so a partial read before
it is written would show), plus the oracle's gate.  The reference call's
workspace is filled with NaN bytes, so a partial it never wrote would show
there too."""
import zlib

import numpy as np
import pytest

from oracle import ops
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

PAIRS = [
    # (first call, second smaller call): N, Ci, Co, D, H, W, k, s, p, bias, dtype
    ((4, 64, 64, 24, 28, 24, 3, 1, 1, True, "bf16"), (2, 64, 64, 12, 14, 12, 3, 1, 1, True, "bf16")),
    ((2, 1, 32, 24, 30, 32, 7, 2, 3, False, "bf16"), (1, 1, 32, 20, 22, 16, 7, 2, 3, False, "bf16")),
    ((2, 64, 64, 4, 8, 16, 1, 1, 0, True, "bf16"), (1, 64, 64, 4, 8, 8, 1, 1, 0, True, "bf16")),
    ((2, 64, 128, 12, 14, 12, 3, 2, 1, False, "bf16"), (1, 64, 128, 6, 7, 6, 3, 2, 1, False, "bf16")),
    ((2, 3, 5, 7, 9, 11, 3, 1, 1, True, "f32"), (1, 3, 5, 5, 5, 5, 3, 1, 1, True, "f32")),
]


def _one(case, accumulate):
    from paper_2104_05035_amd import rat3d as R
    torch = U.torch_mod()
    N, Ci, Co, D, H, W, k, s, p, has_bias, dt = case
    rng = np.random.default_rng(zlib.crc32(repr(case).encode()))
    x, xr = U.dev_input(rng.standard_normal((N, Ci, D, H, W)), dt)
    Do, Ho, Wo = (ops.out_size(v, k, s, p) for v in (D, H, W))
    dy, dyr = U.dev_input(rng.standard_normal((N, Co, Do, Ho, Wo)), dt)
    desc = R.conv_desc(N, Ci, Co, D, H, W, k, s, p, has_bias, U.code(dt))
    need = R.rat3d_conv3d_workspace_size(desc, 2)
    assert need <= R.rat3d_conv3d_wgrad_noalloc_max_bytes()
    ws = torch.full((max(need, 256),), 0xFF, dtype=torch.uint8, device="cuda:0")
    init = torch.from_numpy(rng.standard_normal((Co, Ci, k, k, k)).astype(np.float32)).to("cuda:0")
    binit = torch.from_numpy(rng.standard_normal(Co).astype(np.float32)).to("cuda:0")
    dw_ref, dw = init.clone(), init.clone()
    db_ref, db = (binit.clone(), binit.clone()) if has_bias else (None, None)
    print("noalloc wgrad %s accumulate=%d" % (case, accumulate), flush=True)
    R.rat3d_conv3d_wgrad(desc, x, dy, dw_ref, db_ref, accumulate, ws, ws.numel())
    R.rat3d_conv3d_wgrad_noalloc(desc, x, dy, dw, db, accumulate)
    U.sync()
    assert torch.equal(dw, dw_ref), "dw differs from rat3d_conv3d_wgrad"
    if has_bias:
        assert torch.equal(db, db_ref), "dbias differs from rat3d_conv3d_wgrad"
    dwr, dbr = ops.conv3d_wgrad(xr, dyr, k, s, p, has_bias)
    tw, tb = ops.conv3d_wgrad(np.abs(xr), np.abs(dyr), k, s, p, has_bias)
    base = U.f64(init) if accumulate else 0.0
    U.check(U.f64(dw), dwr + base, dt, "dw", kind="sum", terms=tw + np.abs(base))
    if has_bias:
        bb = U.f64(binit) if accumulate else 0.0
        U.check(U.f64(db), dbr + bb, dt, "db", kind="sum", norm=False, terms=tb + np.abs(bb))


@pytest.mark.parametrize("pair", PAIRS, ids=lambda p: "%dto%d_k%d_%s" % (p[0][1], p[0][2], p[0][6],
                                                                        p[0][10]))
def test_noalloc_wgrad_two_calls(pair):
    first, second = pair
    _one(first, 0)
    _one(second, 1)


def test_noalloc_rejects_oversize():
    """A shape whose partials exceed the built-in scratch is refused before
    anything is enqueued."""
    from paper_2104_05035_amd import rat3d as R
    # a stride-2 conv (split-K gather partials: 3 x 512 x 256 x 27 floats)
    desc = R.conv_desc(8, 256, 512, 12, 14, 12, 3, 2, 1, False, R.BF16)
    assert R.rat3d_conv3d_workspace_size(desc, 2) > R.rat3d_conv3d_wgrad_noalloc_max_bytes()
    fake = 0x10000
    with pytest.raises(R.Rat3dError) as e:
        R.rat3d_conv3d_wgrad_noalloc(desc, fake, fake, fake, None, 0, stream=0)
    assert e.value.status == R.EWORKSPACE
