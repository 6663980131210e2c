"""QuantWM (arxiv 2609.26425) hot path for AMD Instinct MI355X (gfx950).

``paper_2609_26425_amd.quantwm`` binds ``libquantwm.so``: quantize-on-append
(QSAC + INT2 residuals + PSAC) and attention over the packed 2-bit cache, both
as hand-written HIP kernels behind the C ABI in ``include/quantwm.h``.
``paper_2609_26425_amd.build`` compiles the library in-tree.
"""
