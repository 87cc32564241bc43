"""ExFold folded MoE layer for AMD Instinct MI355X (gfx950).

The compute path is the C-ABI library ``libexfold.so`` built from ``csrc/``;
``paper_2608_24938_amd.exfold`` binds it.  Importing the package loads
nothing; the library is loaded on first use and a missing library raises.
"""
