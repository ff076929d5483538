"""CPU oracle for SuperBatch encoding (SURGE, arXiv 2605.01060).

TEST INFRASTRUCTURE ONLY.  The oracle is a plain, slow, float64 NumPy
statement of what the GPU path computes, written from the paper and from the
encoder semantics the paper leaves to its model (see ``encoder``).  Only the
test suite, the smoke check and the benchmark's CPU-baseline leg may import
it; the product package never does, and it imports nothing from the product.

Modules:
  * ``encoder`` - per-text BERT-style encoder forward, masked mean pooling,
    L2 normalisation and partition placement (problem statement, Sec. 2.2;
    Alg. 1 Flush; Sec. 5.1 "L2-normalized embeddings").
  * ``plan``    - SuperBatch aggregation (Alg. 1 AddPartition / Flush, the
    two-threshold trigger of Sec. 3.2 and the oversized-partition split of
    Sec. 6), under the two readings listed in ``plan``'s docstring.

Every function is pinned by a ``-m "not gpu"`` test against something other
than itself: a library encoder (``transformers.BertModel``), brute force on
padded batches, closed forms, invariants and the paper's printed numbers.
"""
