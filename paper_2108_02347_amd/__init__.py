"""FMMformer attention forward on AMD MI355X (gfx950) through hand-written HIP kernels."""
