"""CPU oracle for the split feature-extraction forward pass.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path imports this package:
only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may load it.  It shares no code with the HIP path (``paper_2210_08650_amd``);
the only module both sides use is ``synth`` (seeded random inputs).

``layers`` wraps the plain-C float64 layer definitions in ``oracle.c``;
``models`` assembles them into the frozen feature extractors the paper splits
(Measurement study; Evaluation, Table 2) and runs the forward pass from the
input up to a split layer (Design, "Request flow"; System implementation);
``split`` is Algorithm 1's split-index choice and its competitors.
"""
from . import layers, models, split  # noqa: F401
