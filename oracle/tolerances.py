"""Parity bounds the GPU results are held to against the float64 oracle.

TEST INFRASTRUCTURE ONLY (imported by ``tests/`` and ``__graft_entry__.smoke()``).

* O: max-abs 1e-2 for the computation, plus the bf16 store's own rounding of
  each element (at most 2^-8 |O|), i.e. |O_gpu - O_ref| <= 1e-2 + 2^-8 |O_ref|.
  Rounding O to bf16 alone moves an element by more than 1e-2 once
  |O| > 2.56, which sequences of a few tokens reach (O is then close to a
  single row of V), so a bare 1e-2 cannot be met by any bf16 output there.
* dQ, dK, dV: max |g_gpu - g_ref| <= 2e-2 * max |g_ref| per tensor.
* LSE: max-abs 5e-3.  The forward normalises O by the sum of the same
  bf16-rounded probabilities it multiplies into V (so O is an exact weighted
  mean of V rows), and returns LSE = m + ln of that sum.  Each summand is off
  by at most 2^-8 relative, so the sum is too and |dLSE| <= -ln(1 - 2^-8)
  = 3.9e-3; 5e-3 leaves room for fp32 accumulation.  The backward recomputes
  P = exp(S - LSE) with that same LSE, so its probabilities are normalised
  exactly as the forward's O was.
"""

O_TOL = 1e-2
BF16_U = 2.0 ** -8  # unit roundoff of bf16 (round to nearest even)
GRAD_TOL = 2e-2
LSE_TOL = 5e-3
