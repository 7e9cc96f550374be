"""Tolerance of the MLP-policy outputs, derived from the arithmetic of a device
evaluation rather than fixed by hand.

The oracle's orc_mlp_bounds encloses every value a device evaluation may return
for one observation under an error model with four constants:
* ACC: each fp32 dot product (bias + n products) is off by at most
  ACC * (n + 1) * (|bias| + sum |w x|); 2^-23 is twice fp32's unit roundoff
  per operation, enough for any summation order and rounding direction;
* E_TANH, E_P0: absolute errors of the kernel's tanh and p0 = 1 / (1 + e^d);
* E_LOGPI: error of the kernel's log pi relative to 1 + |log pi|.
The last three are the maxima measured over all 2^32 fp32 inputs of the
kernel's own device functions (tests/test_gpu_policy_math.py: 2.216e-7,
1.108e-7 and 8.464e-8), rounded up.  In bf16 mode the enclosure also follows
every rounding of a hidden unit that the model's errors could move across a
bf16 rounding boundary, which is how a bf16 evaluation can differ from the
oracle's by far more than its fp32 arithmetic would suggest.
"""
import oracle

ACC = 2.0 ** -23
E_TANH = 2.5e-7
E_P0 = 1.25e-7
E_LOGPI = 1.0e-7


def errs(scale: float = 1.0) -> "oracle.Errs":
    """The error model (scale multiplies the three function errors)."""
    return oracle.Errs(ACC, E_TANH * scale, E_P0 * scale, E_LOGPI * scale)
