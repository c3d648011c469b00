"""MI355X-native context-parallel prefill attention (arXiv 2609.04774 hot path).

``paper_2609_04774_amd.cpattn`` is the Python binding of libcpattn (the C ABI
in include/cp_attn.h over hand-written gfx950 HIP kernels);
``paper_2609_04774_amd.build`` compiles that library in-tree;
``paper_2609_04774_amd.calibrate`` fits the attention term of the paper's
prefill-time model (Sec. 3.2) to measured kernel times, and
``paper_2609_04774_amd.placement`` evaluates the adaptive placement cost
(Sec. 5.3) with that model.  Submodules are
imported on first use, so building works before the library exists.
"""

__all__ = ["cpattn", "build", "calibrate", "placement"]


def __getattr__(name):
    if name in ("cpattn", "build", "calibrate", "placement"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
