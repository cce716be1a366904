"""RelaxKV selective-repair hot path on MI355X (gfx950).

The compute path is the HIP library built from ``csrc/``; ``relaxkv`` is its
thin ctypes binding (argument marshalling only).  ``synth`` makes seeded
synthetic inputs.
"""
