"""Independent CPU oracle for prefix-cached paged prefill attention.

This package is TEST INFRASTRUCTURE. Only the test-suite, the smoke check and
the CPU-baseline leg of the benchmark may import it; the product library never
does, and the product path fails loudly when its HIP library is missing rather
than falling back to anything in here.

It shares no code with the HIP/C++ path: no kernels, headers, helpers, tables
or constants are common to both.  Each function states the passage of the
InferLog paper (arXiv 2507.08523) it follows.

* ``prefix_ref``  -- block-level prefix caching with chained block keys
  (paper section 2.1.2, "KV Cache and Prefix Caching", and the figure of three
  requests reusing blocks b1..b3 but not b7, b8).
* ``attn_ref``    -- dense float64 causal grouped-query attention of the
  uncached suffix over cached + new keys (paper section 2.1.2: prefill over the
  prompt, KV of cache-missing tokens computed and stored, section 3.2.2).
* ``pair_ref``    -- prefix-aware refinement of the in-context demonstrations
  and the ICL table (sections 3.2.1 and 3.2.2).
* ``lifecycle_ref`` -- the prefix cache with reference-counted blocks and
  least-recently-used eviction (section 2.1.2).
* ``rope_ref``    -- rotary position embedding of the new tokens' keys and
  queries at their absolute positions (section 2.1.2; RoFormer's rotation).

Readings of points the paper leaves open (block size 16, frozen-snapshot
visibility inside a batch, the fully-cached cap, the hash itself, 1/sqrt(D)
scale, bottom-right causal alignment, contiguous GQA groups) are listed in the
repository's design notes.
"""
