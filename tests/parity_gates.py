"""Tolerances of the GPU parity tests, in one place (imported by them and by
the CPU check that the precision canary is discriminating).

Contract (fp32 output, whole output of a case): max-abs <= 1e-2 and
rel-L2 <= 5e-3.

Precision canary: a regression guard, not the contract.  The kernel's fp32
output sits ~1000x inside the contract gates (max-abs <= 1.1e-5, rel-L2 <=
3e-6 over every case); a weaker softmax/PV path, e.g. the weights P rounded to
bf16 only (no low part), errs ~1e-3 at these lengths and still passes the
contract gates, but not the canary."""
GATE_MAX_ABS = 1e-2
GATE_REL_L2 = 5e-3
CANARY_MAX_ABS = 1e-4
CANARY_REL_L2 = 1e-4
