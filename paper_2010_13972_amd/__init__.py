"""Exact path-based TreeShap on AMD Instinct MI355X (gfx950).

``gts`` is the binding of the C-ABI library ``libgts.so`` (``include/gts.h``);
``synth`` makes the seeded synthetic ensembles used by the tests and the
benchmark.
"""
from . import gts, synth  # noqa: F401
from .gts import (DeviceModel, GtsError, extract_paths, model_layout, pack_paths,  # noqa: F401
                  prepare, shap, shap_interactions)
