"""MI355X-native INT4 RotateAttention: HIP kernels for gfx950 behind a C ABI.

The binding (``paper_2607_02584_amd.rotate_attn``) loads ``librotate_attn.so``
lazily; importing the package itself loads nothing.
"""
__all__ = ["datagen", "rotate_attn"]
