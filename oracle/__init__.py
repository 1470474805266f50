"""CPU oracle of the sparse-KV decode hot path.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only tests, the smoke check and
the benchmark's CPU-baseline leg may import it.  Shares no code with the GPU
package (paper_2609_34555_amd).
"""
