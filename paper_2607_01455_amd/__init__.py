"""Ember token-table optimizer step for AMD MI355X (gfx950).

``paper_2607_01455_amd.ember`` is the binding of the HIP library libember.so
(C ABI in include/ember.h); importing it fails if the library is not built.
``paper_2607_01455_amd.workloads`` holds seeded synthetic inputs.
"""


def __getattr__(name):
    if name in ("ember", "workloads", "build"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
