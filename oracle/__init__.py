"""CPU oracle for tree verification over CSA/HCA compressed attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the library's product path may import,
call or execute this package: only the test suite, the smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code with the GPU library.

``tv_oracle`` computes the four steps (ancestor mask, per-branch compression,
verify attention, accepted-path commit) directly on the tree, in float64.
``replay`` decodes every root-to-leaf branch as an independent linear sequence;
the tree result must equal it node by node.
"""
from . import tv_oracle  # noqa: F401
from . import replay  # noqa: F401
