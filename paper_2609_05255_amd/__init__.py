"""MI355X-native differentiable Gaussian-splatting rasterizer with fused SH3 or
latent+MLP appearance (Compact Neural Appearance Models for Efficient Gaussian
Splatting). The GPU work lives in the HIP library ``libgsraster.so`` behind the
C ABI of ``include/gsraster.h``; ``gsraster`` is its Python binding and
``inputs`` the seeded synthetic-input generator."""

__version__ = "0.1.0"
