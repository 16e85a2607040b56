"""MI355X-native PRECOG hot path: gated selective-SSM prefill scan with an
injectable initial state and captured final state, cosine top-1 retrieval and
state-injection gather, as hand-written gfx950 HIP kernels behind the C ABI
declared in ``include/precog.h``.

The binding (``paper_2608_02560_amd.precog``) is imported lazily so that the
input generators (``paper_2608_02560_amd.synth``) can be used without loading
the HIP library.
"""

__all__ = ["precog", "synth"]


def __getattr__(name):
    if name in __all__:
        import importlib

        return importlib.import_module(__name__ + "." + name)
    raise AttributeError(name)
