"""CPU oracle for the population-decode hot path (TEST INFRASTRUCTURE ONLY).

A plain, slow, obviously correct fp64 NumPy statement of what the GPU path
computes.  Only the tests, ``__graft_entry__.smoke()`` and the bench's
``cpu_baseline`` leg may import it; the product library never does, and this
package imports nothing from it.  It shares no code with the HIP path: the
only module both sides use is ``workload`` (seeded inputs, no method
arithmetic).

Contents and the passages each part follows:

* ``formats``   - bf16 and OCP E4M3FN decoding to fp64 (storage formats of
                  the KV cache; the fp8 per-block scale follows the workload
                  definition of the fp8 configuration), and the E4M3FN
                  encoding of quantise-on-append (nearest value, ties to the
                  even code, saturating; the quotient x / scale in fp32).
* ``attention`` - decode-step attention of one trace over its whole context,
                  the plain softmax(q K^T * s) V definition with grouped KV
                  heads.  The method's saving is that children inherit the
                  parent's KV (Alg. 1 notation, Branch; Sec. 4.1 Case 2;
                  Sec. 5.3), which changes where the KV lives, not the
                  result, so the oracle computes on materialised per-trace
                  copies.
* ``probe``     - the linear sigmoid probe sigma(w.h + b) (the head form of
                  Eq. 6 applied to h), ranking by score descending with ties
                  to the lowest trace id (Alg. 1 Tournament: rank, bottom-K
                  prune, top-K branch; Eqs. 2-3), and the prune/branch plan.
* ``pool``      - an independent model of the refcounted paged KV pool:
                  lowest-free-first block allocation, fork = share full
                  blocks + copy the partial tail, free = drop references
                  (Sec. 4.1 Case 2: pruning frees the non-shared blocks, the
                  child reuses its parent's KV by prefix caching);
                  a decode step's bf16 K/V quantised into fp8 blocks with the
                  landing block's scale.
* ``tournament`` - the full tournament of Alg. 1 over the pool model:
                  running-mean scores, GenLen eligibility, Case 1 fill
                  (Eq. 2), Case 2 swap (Eq. 3), scheduler eviction of the
                  lowest-scoring running trace into a ghost that keeps its
                  place in the tree view (Sec. 4.2).
* ``mlp``       - the 2-layer MLP scorer sigmoid(w2 . act(W1 h + b1) + b2)
                  (the paper's main-evaluation scorer family, Sec. 5.1;
                  dimensions, activation and weights are parameters).
* ``seqscorer`` - the history-aware sequence scorer of App. A.1 (Eqs. 4-6):
                  input LN, W_in, GELU, pre-norm causal Transformer layers
                  (RoPE attention, SwiGLU), output LN, w_out, sigmoid; the
                  whole history recomputed at every boundary.

Parity status: every function is pinned by the ``-m "not gpu"`` tests
(closed forms, library special cases, invariants, brute force, exhaustive
code tables, hand-worked block counts, torch's LayerNorm / GELU / SiLU /
causal scaled-dot-product attention).  The paper prints no numeric example
of attention, scores or block tables, so no pin is a value from the paper.
"""
