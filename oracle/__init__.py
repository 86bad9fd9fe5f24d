"""CPU oracle for the AtSpeed verify path (arXiv 2410.05165).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 implementation
of what the GPU path computes, written from the paper's definitions.  Only the
test suite, the smoke check of ``__graft_entry__`` and the ``cpu_baseline``
leg of ``bench.py`` may import it; the product library never does, and the
oracle shares no code with the HIP path.

Modules
  numerics  bf16 rounding emulation and bf16 decoding (fp64 arithmetic)
  model     LLaMA-style causal decoder (one forward per path; optional explicit
            attention mask for the flattened-tree form)
  trie      item-identifier prefix trie (plain dict of sets)
  tree      flattening of drafted beams into a tree with an ancestor mask
  search    target-only constrained beam search, draft beam search,
            strict top-K verification (Algorithm 1), speculative decode loop
  philox    Philox4x32-10 counter-based generator (Salmon et al., SC'11)
  relaxed   relaxed sampling verification (Sec. 3.2, Algorithm 2)
  align     draft alignment objectives AtSpeed-S / AtSpeed-R (Sec. 3.1, 3.2),
            their gradients and the item-head gradient

Parity status of each function is stated in its module docstring.
"""
