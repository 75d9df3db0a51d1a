"""Plain float64 CPU oracle for the GLANCE decode-round hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and its
Python binding) may import, call or link anything here; only the test suite,
the smoke check and the CPU-baseline leg of the benchmark use it.

The oracle is written from the paper (arXiv 2609.00355) and shares no code with
the GPU path:

* ``attention``  -- explicit-mask softmax attention for the one-pass block draft
  (Sec. 3.2, "One-Pass Drafting on Fused States") and the ancestor-masked
  tree verification (Def. 1, Sec. 3.3; Algorithm 1 "pack b and T with an
  ancestor mask", App. B);
* ``accept``     -- per-row vocabulary argmax and the greedy walk of Algorithm 1
  (App. B), plus an independent evaluation of the accepted length
  A(T) = max{k : Y_{1:j} in T for all j <= k} of Def. 1;
* ``commit``     -- the commit of a round's accepted path: the keys and values of
  the root and the accepted nodes join the context cache (Def. 1's walk
  commits them; Eq. 1);
* ``sampling``   -- the walk at temperature T > 0: each visited row's draw by the
  Gumbel-max rule with Philox4x32-10 uniforms and a fixed fp32 logarithm;
* ``tree``       -- the tree builder of Sec. 3.3 (Algorithm 1, second step): the
  N strings of highest plug-in score prod_j q_j(y_j) (Assumption 1) packed as
  a prefix-closed tree, by exhaustive and by best-first enumeration;
* ``tiny_model`` -- a tiny random-weight float64 decoder used to check the
  lossless greedy equivalence of Thm. 1 (Sec. 3.3, App. A.1).
"""

from . import attention, accept, commit, sampling, tiny_model, tree  # noqa: F401
