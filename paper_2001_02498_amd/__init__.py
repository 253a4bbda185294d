"""MI355X-native subgraph GCN training hot path (GraphACT, FPGA '20).

Importing the package loads nothing native; `paper_2001_02498_amd.gcn` loads
the HIP library on first use and raises if it is missing.
"""
