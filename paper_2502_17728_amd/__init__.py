"""Deferred normalization on MI355X (gfx950).

LayerNorm -> Linear and Softmax -> P.V with the normalization deferred past
the matrix product, after "LLM Inference Acceleration via Efficient Operation
Fusion" (arXiv 2502.17728), Sec. II-A (Eq. 5) and Sec. II-B (Eq. 8).

Importing the package loads nothing native.  ``paper_2502_17728_amd.ops``
loads the HIP library (``libdn.so``) and raises if it is missing;
``paper_2502_17728_amd.inputs`` holds the seeded synthetic workloads.
"""

__all__ = ["ops", "inputs", "build"]
__version__ = "0.1.0"


def __getattr__(name):
    if name in ("ops", "inputs", "build"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
