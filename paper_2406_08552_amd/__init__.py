"""DiTFastAttn attention hot path on AMD MI355X (gfx950).

The compute path is the C-ABI library ``libdfa.so`` built from ``csrc/``;
``paper_2406_08552_amd.dfa`` is its thin ctypes binding.  Importing this
package loads nothing; ``inputs`` holds the seeded synthetic input generator.
"""
__all__ = ["dfa", "inputs"]
