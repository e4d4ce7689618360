"""The device input generator reproduces the host generator bit for bit."""
import numpy as np
import pytest

from synth import workloads as wl

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_device_generator_matches_host(dtype):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import synth.device as sdev
    w = wl.RAGGED32.replace(dtype=dtype)
    for spec in (wl.spec_h(w, 3), wl.spec_q(w, 5), wl.spec_kv_direct(w, "v", 7, 100, 333),
                 wl.spec_wf(w)):
        g = sdev.materialise(w, spec).cpu()
        h = wl.host_block(w, spec)
        if dtype == "bf16":
            np.testing.assert_array_equal(g.view(torch.int16).numpy().view(np.uint16), h)
        else:
            np.testing.assert_array_equal(g.numpy(), h)
