"""QUAN hot path on MI355X (gfx950): the quaternion (Hamilton-product) 2-D
convolution and Independent Quaternion Batch Normalization, as hand-written HIP
kernels behind a C ABI (libquan.so).  ``quan`` is the thin ctypes binding;
``workloads`` draws the seeded synthetic inputs."""
