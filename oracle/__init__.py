"""Float64 CPU oracle for one reverse step of a discrete-diffusion language model.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package: only the test suite, the smoke check and the
CPU-baseline leg of the benchmark use it.  It shares no code, constants or
helpers with the HIP library; both sides implement the counter-based generator
(Philox4x32-10) from its published definition.

Modules, each written from the paper (arXiv 2609.04010) and cited per function:

  philox     Philox4x32-10 (Salmon et al., SC'11), vectorised and scalar
  noise      uniform / exponential / Gumbel / normal transforms of a word
  schedule   alpha_t = 1 - t and the grid t_k = k/T
  params     parameter list and seeded initialisation
  forward    the bidirectional transformer denoiser x_theta(z_t, t)
  forward_loops  the same denoiser written as scalar loops (pin of forward)
  posterior  masked / uniform-state reverse posteriors and the Psi forms
  bayes      brute-force enumeration of the forward process (pin)
  sampler    two-level Gumbel-max categorical sampling
  latent     Gaussian-latent argmax and the alpha_tilde <-> alpha map
  loop       the T-step ancestral sampling loop

Parity status of each function is listed in its module header; the forward
pass has no paper-fixed values and is pinned by invariants and by a second
independent implementation.
"""
