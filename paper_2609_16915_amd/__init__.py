"""Batched TFHE programmable bootstrapping (ROSETTA's nonlinear-layer hot
path) on AMD Instinct MI355X: HIP kernels behind a C ABI (librosetta.so),
with a thin ctypes binding in `rosetta` and seeded workloads in `workloads`."""
