"""Oracle for the cache-hit generation path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, CPU-only (NumPy) statement of what the path computes, written
from the paper's definitions:
  lookup.py    cosine top-1 over cached prompt embeddings and the similarity
               -> K selector (Sec. 4.3 Alg. 1, Sec. 5.3.1 cache selector);
  schedule.py  the DDIM timestep grid and cumulative alpha table (Sec. 2.1, Sec. 6);
  ddim.py      classifier-free guidance and the deterministic DDIM update, and the
               resume-from-step-K loop of approximate caching (Sec. 4.1);
  unet.py      the latent-diffusion UNet epsilon predictor (Sec. 2.1), fp32;
  lcbfu.py     cache maintenance under LCBFU and the hole-aware choice of the
               state served (Sec. 5.4);
  predictor.py the match predictor, a linear one-class SVM trained by SGD
               (Sec. 5.2, Sec. 6);
  ivf.py       an inverted-file approximate index over the cached embeddings
               (the indexed vector-DB search of Sec. 5.3 / Sec. 6).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package.  The product path never imports it and shares no code with it.
"""
