"""CPU oracle for Approximate Random Dropout (Song et al., arXiv 1805.08939).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call, link or
execute this package: only the test suite, the smoke check of the package entry
point, and the CPU-baseline leg of the benchmark use it.

The oracle is a plain, slow, obviously correct restatement of what the method
computes, written from the paper:

* ``prng``     - the counter-based generator (SplitMix64) and the per-iteration
                 pattern sampler of Sec. III-D, plus tile bitmaps (Sec. III-B).
* ``patterns`` - row-based (Sec. III-A, Eq. 1) and tile-based (Sec. III-B)
                 dropout patterns as masks and as ascending gather lists.
* ``search``   - the SGD-based search for the pattern distribution K
                 (Sec. III-C, Alg. 1): the paper's gradient iteration and the
                 closed-form minimiser of its loss.
* ``fc``       - a fully connected layer under a row pattern, as a dense fp64
                 GEMM with the dropout mask multiplied in (Sec. II-C, Sec. III-A).
* ``tdp``      - a layer under a tile pattern (Sec. III-B), dense with the tile
                 mask multiplied in.
* ``lstm``     - an LSTM layer whose hidden units follow a row pattern fixed per
                 sequence, with manual back-propagation through time (Sec. IV-C).

Floating point is fp64 throughout. The oracle shares no code with the HIP
library: it reads only numpy (and pure Python integers for the generator).
"""
