"""MI355X-native routed MoE FFN forward (EPS-MoE hot path).

The compute path is the HIP library ``libmoe.so`` built from ``csrc/``; the
Python side only marshals arguments (see ``moe``).  Importing this package
loads nothing: ``moe`` loads the library on first use and raises if it is
missing.
"""
