"""GRIFFIN-style tree verification on AMD Instinct MI355X (gfx950).

The verify pass (target model over a draft tree, greedy acceptance walk) runs
entirely in the HIP library libgriffin_verify.so behind the C ABI of
include/griffin_verify.h; this package is its Python binding.  The library is
loaded on first use of any binding name (so that `paper_2502_11018_amd.build`
can run without it) and its absence raises ImportError.
"""

_EXPORTS = {
    "AcceptResult": "verifier", "TreeVerifier": "verifier", "accept_walk": "verifier", "accept_sampled_walk": "verifier", "pack_trees": "verifier",
    "tree_prepare": "verifier", "GriffinError": "_native", "STATUS": "_native", "KERNEL_CLASSES": "_native",
    "DraftModel": "draft", "SpeculativeCycle": "cycle",
}


def __getattr__(name):
    if name in _EXPORTS:
        import importlib
        mod = importlib.import_module(f".{_EXPORTS[name]}", __name__)
        return getattr(mod, name)
    raise AttributeError(name)


__all__ = sorted(_EXPORTS)
