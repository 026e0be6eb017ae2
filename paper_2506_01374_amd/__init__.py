"""MI355X-native schedule-parameterised contractions (the operator family that
the Reasoning Compiler searches over), a C-ABI library around them, a timing
harness and a UCT / random schedule search.

Importing the package loads nothing native; ``paper_2506_01374_amd.rc`` loads
``librc.so`` on first use and raises if it is missing.
"""
__all__ = ["inputs", "rc"]
