"""RoLA sparse + rotary-low-rank attention for AMD Instinct MI355X (gfx950).

The compute path is the HIP library `librola.so` behind the C ABI declared in include/rola.h;
`paper_2609_06712_amd.rola` is its thin ctypes binding and `paper_2609_06712_amd.synth` draws seeded
synthetic inputs. Importing the package itself loads nothing.
"""
