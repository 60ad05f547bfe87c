"""CPU oracle for LoopSpec (pipelined self-speculative decoding of Looped
Transformers): plain, slow, fp64 reference code written from the paper.

TEST INFRASTRUCTURE.  Only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg may import, call or execute anything in this package.  It
shares no code with the HIP path (paper_2609_17184_amd); both only read the
seeded synthetic inputs of the `synth` module.

Modules
  model     fp64 looped forward (per-depth KV caches) and a cache-free recompute
  dist      readout distributions (T, top-p), residual operator, TV, draws
  philox    Philox4x64-10 keyed draws (pinned against numpy.random.Philox)
  loopspec  Alg. 1 simulator and vanilla looped decoding
  theory    Theorem 1/2 tools, envelope fit, branch growth, gamma

Pins (tests/test_oracle_*.py) tie each module to something other than itself:
values printed in the paper, closed forms, exact enumeration, invariants and
independent library routines.  Nothing here is "parity unpinned".
"""
from . import dist, loopspec, model, philox, theory   # noqa: F401
