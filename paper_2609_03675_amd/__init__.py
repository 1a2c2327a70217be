"""CoFiE evidence selection (NGFF + QER) on MI355X: HIP kernels behind a C ABI."""
