"""CPU oracle for SDQ-LLM (arXiv 2510.03275): TEST INFRASTRUCTURE ONLY.

A plain, slow, step-by-step CPU implementation of what the hot path computes,
written from the paper and used to check the HIP library.  Only the tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it; the product path (``paper_2510_03275_amd``) never does, and the two
share no code.

Contents (each function cites the passage it follows):

* ``hadamard``    -- Sylvester Hadamard matrices (Section 3.3, Eq. 13), the
                     fp32 fast Walsh-Hadamard transform used for block smoothing,
                     and the choices of Had (Sylvester, sign-randomised, none);
* ``resample``    -- the FFT ``Resample`` function of Algorithm 1 and the
                     closed forms of its up- and down-sampling matrices;
* ``sigma_delta`` -- the binary / ternary quantizers (Eq. 3-6) and the
                     first-order Sigma-Delta recursion (Eq. 7-8);
* ``encoder``     -- weight encoding: block Hadamard, Resample up, per-row
                     scale, Sigma-Delta scan (Algorithm 1, ``SDQuant``);
* ``linear``      -- the fp64 plain definition y = x W_hat^T of the
                     dequantized linear (Algorithm 1's reconstruction,
                     Fig. 5) and the activation-expansion identity;
* ``layout``      -- the packed code format of the library's C header,
                     re-implemented independently, and Eq. 14's ratio;
* ``multiosr``    -- the per-linear OSR allocation of Section 3.4 (reading
                     documented in the module; parity of its exact rule is
                     unpinned by the paper);
* ``compensation``-- the block compensation of Algorithm 1 (Hessian, the
                     Cholesky factor of its inverse, the block loop).

Precision: the encoder runs in fp32 with every multiply and add rounded
separately (no fused multiply-add), so its codes are a bit-exact target; the
linear and everything else run in fp64.
"""
from . import hadamard, resample, sigma_delta, encoder, linear, layout, multiosr, compensation  # noqa: F401
from .encoder import encode, EncodeResult  # noqa: F401
from .linear import linear_fp64, reconstruct_fp64, expand_activations_fp64  # noqa: F401
from .multiosr import variance_fp64  # noqa: F401
