"""MI355X-native ProtoKV far-memory hot path (libprotokv + thin binding).

Importing the package loads nothing; ``paper_2606_26762_amd.protokv`` loads
the HIP library on first use and raises if it is missing.
"""
