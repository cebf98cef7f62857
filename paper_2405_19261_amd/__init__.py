"""libspeccascade: the verify/defer step of speculative cascades on MI355X (gfx950).

``paper_2405_19261_amd.spc`` binds the C interface of ``libspeccascade.so``
(declared in ``include/speccascade.h``); ``paper_2405_19261_amd.workloads``
draws seeded synthetic inputs.  Importing the package loads nothing native;
the shared library is opened on first use and a missing build is an error.
"""
__all__ = ["spc", "workloads"]
