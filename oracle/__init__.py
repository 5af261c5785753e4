"""CPU oracle for byte-exact KV-state grafting -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline leg
may import anything from here.  The product path (``paper_2607_14431_amd``)
never does, and this package never imports the product path: the two share no
code.  Both draw their raw inputs from the seeded generator in ``synth``.

What it computes, each in plain numpy (fp64 unless a storage rounding says
otherwise), from the paper's statement of the method:

* ``rope``       rotary position embedding of q/k at absolute positions and the
                 re-rotation of a relocated block (RoFormer rotary encoding, used
                 by the paper's model; relocation, Sec. 4.2).
* ``numerics``   round-to-nearest-even to the storage dtype (bf16 / fp32).
* ``paging``     a paged KV pool addressed through block tables; the deposit
                 (state capture) as a gather of a prefix's pages into one
                 contiguous payload, the graft (state restore) as the inverse
                 scatter (Sec. 3.1-3.2).
* ``attention``  causal grouped-query softmax attention for query rows at given
                 logical indices (fresh-context inference on top of the restored
                 prefix, Sec. 3.2; decode over the restored context, Sec. 4.3).
* ``path``       the fresh computation of a workload end to end, whose outputs
                 the graft path must reproduce byte for byte (Eq. 1).
* ``digest``     SHA-256 content digests of an artifact's leaves, a Merkle root over
                 them and the content-addressed dedup map (block digests, Sec. 4.11).
* ``logits``     a synthetic soft-capped logit head over the hidden vector, the KL
                 divergence and argmax of two logit vectors, and the Mann-Whitney U /
                 Cliff's delta statistics of the exactness test (Eq. 1-2, Sec. 4.1-4.2).

Pins (tests marked ``not gpu``): Philox known-answer vectors, literal RoPE
values, rotation-group identities, brute-force attention loops and closed
forms, gather/scatter round trips and block-table permutation invariance, the
published FIPS 180 SHA-256 examples and brute-force dedup on raw leaf bytes, the
soft cap's tanh closed form and limits, two-point KL closed forms and scipy's
Mann-Whitney test.  The magnitudes of the paper's nonzero KL figures (relocated
blocks, cross-engine replays) need its trained model and are not reproduced; the
exact-graft statistics (KL 0, equal argmax, p = 1, delta = 0) are.
"""
