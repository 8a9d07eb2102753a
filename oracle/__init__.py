"""The oracle: a plain, slow CPU statement of the BaryCache hot path.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the benchmark's CPU
baseline leg may import anything from this package; the product path never
does.  It shares no code with the HIP library (paper_2608_28670_amd).

  bary    -- barycentric weights (Sec. 3.2, Eqs. 8-12), full/forecast mask,
             cache ring and per-step plan, forecast (Eq. 13)
  model   -- the DiT-family denoiser (Sec. 3.1, Eqs. 4-5)
  sampler -- schedules, sampler updates and the sampling loop (Sec. 3.3)
"""
from . import bary, model, sampler  # noqa: F401
