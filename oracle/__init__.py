"""Oracle: a plain, slow CPU fp64 implementation of one generation of the
spatial coevolutionary GAN training the paper describes (Section 3,
"Coevolutionary GAN Training", steps 1-5).

THIS IS TEST INFRASTRUCTURE.  Only the tests, the smoke check of the entry
module and the CPU-baseline leg of the benchmark may import it.  It shares no
code with the HIP path: the only inputs the two have in common are the seeded
workloads and datasets of the ``synth`` package, and the random numbers both
sides draw from their own implementations of Philox4x32-10.

Modules
  rng      Philox4x32-10 and the uniform / normal / index draws made from it
  grid     toroidal grid and 5-cell von Neumann neighbourhoods
  mlp      MLP forward / manual backward in fp64, flat parameter layout, init
  dcgan    DCGAN-style conv / transposed-conv / batch-norm networks, forward
           and manual backward in fp64, flat parameter layout, init
  coevo    state, evaluation, fitness, tournament, replacement, mutation,
           training step (Adam), one generation
  mixture  the (1+1)-ES over the generator-mixture weights and its score
  nes      the gradient-free NES trainer (antithetic estimate + Adam)
  es       the gradient-free (1+lambda)-ES trainer (plus-selection over
           antithetic Gaussian mutants)

Pinned by tests/test_oracle_*.py against: published Philox known-answer
vectors and rocRAND's host Philox, hand-enumerated neighbourhoods, BCE closed
forms, finite differences, torch CPU fp64 convolutions, batch norm and autograd, Adam closed forms and
torch.optim.Adam, brute-force tournament enumeration, the 1x1-grid reduction
to plain alternating GAN training, Frechet-distance closed forms, the
mixture's generator moments recomputed with torch fp64 layers on the shared
latents and the closed form of a constant generator, and, for
NES, exactness on quadratics and convergence to the backpropagated gradient;
for ES, the selection rule on hand-made losses, brute-force scoring of every
candidate with torch networks and the elitist invariant; for sub-populations,
uniform tournament draws over ordered tuples, members that train exactly like
the cells of a wider grid, an evaluation that scores every pair of the
neighbourhood population, and the elitist truncation on hand-made fitness
lists.

Parity unpinned: trajectories over many steps or generations at workload
scale.  The paper prints no worked values for them, and the GAN dynamics
amplify any rounding (a run differing from another by one fp32 rounding of
its start state ends 7e-4 apart after 100 steps), so they are compared with
the GPU only step by step from shared states.
"""
