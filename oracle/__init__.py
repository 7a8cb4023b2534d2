"""CPU oracle for the diffusion denoise loop and the approximate-cache lookup.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import,
call or execute anything in this package. The product path (the C-ABI library
and its Python binding) never routes through it and shares no code with it.

What it computes (Argus, arXiv 2511.06724):

* the approximate-caching (AC) worker step of Sec. 2.1 and Sec. 4.5/4.7: find
  the cached prompt whose embedding is nearest to the query, take its
  intermediate latent at iteration K and finish the remaining N-K denoising
  iterations with the new prompt;
* each iteration is one evaluation of the latent-diffusion UNet (the component
  Table 3 and Observation 5 of Sec. 3.2 identify as the compute-bound part of
  generation) with classifier-free guidance, followed by a deterministic DDIM
  update.

The paper names the models (SD-XL, SD 1.5/2.0, Tiny/Small SD) but not their
internals, so every formula here is the public definition of the named method:
DDIM (Song, Meng & Ermon 2021), classifier-free guidance (Ho & Salimans 2022),
the latent-diffusion UNet (Rombach et al. 2022; SD-XL: Podell et al. 2023),
GroupNorm (Wu & He 2018), GEGLU (Shazeer 2020). Each function's docstring names
the definition it follows.

Precision: fp32 tensors for the UNet (as the published models run), fp64 for
the noise schedule and the cosine scores. Parity of the whole UNet on random
weights is pinned only through its parts (see ``tests/test_oracle_*``): each
primitive is checked against brute force, closed forms or invariants, and the
topology against the parameter and FLOP counts of Table 3.
"""

from . import layers, schedule, topology, unet, sampler, lookup  # noqa: F401
