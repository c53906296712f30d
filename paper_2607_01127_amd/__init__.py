"""LogbQuant 4-bit weight-only inference on AMD MI355X (gfx950).

``paper_2607_01127_amd.logbq`` binds the C ABI of ``liblogbq.so`` (include/logbq.h);
``paper_2607_01127_amd.inputs`` draws the seeded synthetic workloads;
``paper_2607_01127_amd.build`` compiles the library in-tree.
"""
