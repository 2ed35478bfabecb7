"""ASAP stochastic-reduce hot path for MI355X (gfx950).

Many logical workers share one GPU.  Each round every worker runs a local
minibatch SGD pass on its own shard, then the stochastic reduce mixes each
worker's model with its in-neighbours' models over a doubly-stochastic
communication graph (Appendix A, update equation (A.2)).  The compute lives in
the C-ABI library ``libasap.so`` (hand-written HIP kernels); ``asap`` is its
thin Python binding and ``synth`` draws the seeded synthetic inputs.
"""
