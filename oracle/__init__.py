"""CPU oracle for the FastCHGNet training step (test infrastructure only).

This package is the plain, slow reference that the GPU path is checked
against. It is written from the paper's definitions, in NumPy float64 (the
neighbour-list predicate alone is evaluated in float32, as the method's
inclusion test is defined on fp32 inputs), with the GatedMLPs applied to the
literal concatenated inputs and a hand-written first-order backward.

Only the test suite, the entry point's smoke check and the benchmark's CPU
baseline leg may import it. It shares no code with the GPU library and the
GPU library never calls it.

Modules:
    graph  - periodic atom graph, bond graph and angle list (Sec. II-B (1)).
    model  - parameter layout, basis expansions, embeddings, interaction
             blocks in the dependency-free form, Force/Stress/Energy heads,
             loss, backward for every parameter, Adam.
    md     - velocity-Verlet molecular dynamics with the model's forces.
    autodiff - an independent PyTorch fp64 transcription of the forward,
             differentiated by autograd: a witness of the hand-written
             backward and the training gradient through the conservative
             readout (second derivatives).
"""
from . import graph, model  # noqa: F401
