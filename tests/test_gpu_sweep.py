"""GPU parity of the single-layer channel sweep (one 3x3 stride-1 conv,
Cin in {16, 32, 64, 128} x Cout in {8, 16, 32, 64, 128}) on the 504 x 504
forward-looking drone stream, against the CPU oracle: change lists bit for
bit at every stride, maps within 1e-4 * max|ref| (fp32)."""
import pytest

import streams as S
from gpu_util import note, run_stream

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

SHAPES = [(ci, co) for ci in S.SWEEP_CIN for co in S.SWEEP_COUT]


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu-test] start {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def test_l64x64_100_strides():
    """The paper's highlighted shape (64 -> 64) over the full 100 strides."""
    run_stream("l64x64", map_every=20)


@pytest.mark.parametrize("cin,cout", SHAPES)
def test_every_sweep_shape(cin, cout):
    run_stream(f"l{cin}x{cout}", n_strides=12, map_every=6)
