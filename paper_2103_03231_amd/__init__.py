"""DONeRF per-ray inference on MI355X (gfx950): a HIP library behind a C ABI
(``include/donerf.h``) and a thin ctypes binding (``paper_2103_03231_amd.binding``)."""
