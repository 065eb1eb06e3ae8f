"""hcmix: the rotating-hypercube mixing layer stack on AMD Instinct MI355X (gfx950).

Importing the package loads nothing native; ``paper_2609_18145_amd.hcmix``
loads the HIP library on first use and raises if it is missing.
"""
