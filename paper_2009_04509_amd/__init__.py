"""MI355X-native per-hit track/shower/Michel classification (arXiv:2009.04509).

The compute path is the HIP library ``libpointid.so`` built from ``csrc/``
(``python -m paper_2009_04509_amd.build``); ``binding`` is its ctypes binding.
Attributes of the binding are re-exported lazily, so that the build script can
be imported before the library exists; touching any of them without the
library raises ImportError.
"""

__all__ = [
    "pointid_create", "pointid_destroy", "pointid_classify", "pointid_classify_planes",
    "pointid_classify_patches", "pointid_gather", "pointid_gather_planes",
    "pointid_last_error", "pointid_version", "PointIdError", "Handle",
]


def __getattr__(name):
    if name in __all__ or name in ("binding", "lib"):
        import importlib
        binding = importlib.import_module(__name__ + ".binding")
        return binding if name == "binding" else getattr(binding, name)
    raise AttributeError(name)
