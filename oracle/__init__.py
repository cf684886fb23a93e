"""Plain CPU float64 oracle for SCOOT's candidate-scoring step (arXiv 2408.04323).

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The product path
(``paper_2408_04323_amd``) never imports it, and this package never imports the
product path: the two share no code.  The only inputs both see come from the
seeded generators in ``workloads``, which hold none of the method's arithmetic.

Each function follows a passage of the paper (SCOOT: SLO-Oriented Performance
Tuning for LLM Inference Engines) and is written for clarity, not speed:

* ``gp``          -- GP surrogate, posterior mean and variance (Sec. 4.3, Eq. 4-5)
* ``acquisition`` -- expected improvement (Sec. 4.4.1, Eq. 8)
* ``hypervolume`` -- hypervolume, its improvement and EHVI (Sec. 4.4.2, Eq. 9, Fig. 4)
* ``forest``      -- random-forest probability of feasibility and the
                     POF >= Delta mask (Sec. 4.7, Eq. 3)
* ``forest_train``-- training the feasibility forest: exhaustive regression
                     trees on SplitMix64 bootstrap samples (Sec. 4.7)
* ``select``      -- top-k parallel suggestion (Sec. 4.6)
* ``threshold``   -- adaptation of Delta (Algorithm 1, Sec. 4.7)
* ``believer``    -- sequential Kriging-believer picks (not in the paper; an
                     extension of the parallel suggestion of Sec. 4.6)
* ``mle``         -- maximum-likelihood GP hyperparameters (Sec. 4.3)
* ``sobol``       -- candidate generation: Sobol pool on the space's grids, known
                     constraints (Sec. 4.5.3, 4.7, Algorithm 1)
* ``mace``        -- MACE for one objective: UCB, PI, EI (Eq. 6-8), their Pareto
                     front over the pool and a seeded random pick (Sec. 4.5.1, 4.6)
* ``pipeline``    -- the whole scoring pass over a candidate pool
* ``suggest``     -- the suggestion step of Algorithm 1 end to end: learn,
                     train, generate, score, pick, fill

Conventions (the readings of the paper this oracle takes):

* every objective is minimised; a caller maps the paper's maximisation of
  lambda * f (Eq. 1) by passing y = -lambda * f;
* the covariance is Matern-5/2 with one lengthscale per dimension (ARD); the
  paper's own kernel is Matern-3/2 with input warping (Sec. 4.3);
* the variance is that of the latent f (Eq. 5 writes sigma^2(f(x))), clamped
  at zero against rounding.
"""
