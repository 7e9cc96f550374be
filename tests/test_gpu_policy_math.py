"""The policy kernel's elementwise functions, measured at every fp32 input.

rlsim_probe_policy_math evaluates the kernel's own tanh, p0 and log pi device
functions at all 2^32 fp32 bit patterns (NaN and infinities skipped) against
double precision.  The maxima must stay within the elementwise error constants
that the policy tolerance (tests/policy_bounds.py) is built on."""
import pytest

import policy_bounds

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _measure(lo, count):
    from paper_2207_07736_amd.probe import probe_policy_math
    out = torch.zeros(3, dtype=torch.int32, device="cuda")
    probe_policy_math(lo, count, out)
    torch.cuda.synchronize()
    return [float(v) for v in out.view(torch.float32).cpu()]


def test_elementwise_errors_over_every_fp32_input():
    e_tanh, e_p0, e_lp = _measure(0, 1 << 32)
    print(f"measured: tanh {e_tanh:.4g}  p0 {e_p0:.4g}  log pi {e_lp:.4g} (relative to 1 + |log pi|)", flush=True)
    assert 0.0 < e_tanh <= policy_bounds.E_TANH
    assert 0.0 < e_p0 <= policy_bounds.E_P0
    assert 0.0 < e_lp <= policy_bounds.E_LOGPI


def test_probe_merges_ranges_and_rejects_bad_arguments():
    from paper_2207_07736_amd.probe import probe_policy_math
    # [0.5, 2): the maxima over the halves merge to the maximum over the whole
    lo, mid, hi = 0x3F000000, 0x3F800000, 0x40000000
    whole = _measure(lo, hi - lo)
    out = torch.zeros(3, dtype=torch.int32, device="cuda")
    probe_policy_math(lo, mid - lo, out)
    probe_policy_math(mid, hi - mid, out)
    torch.cuda.synchronize()
    assert [float(v) for v in out.view(torch.float32).cpu()] == whole
    for args in ((0, 0, out), (1, 1 << 32, out), (0, 4, None)):
        with pytest.raises(ValueError):
            probe_policy_math(*args)
