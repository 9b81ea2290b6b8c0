"""Memoized DNN mutation testing on AMD Instinct MI355X (gfx950).

The work happens in ``libmure.so`` (HIP kernels behind the C ABI of
``include/mure.h``); this package is its Python binding.
"""
from .binding import (Mure, MureError, load_library, LIB_PATH, EXPORTED,
                      MURE_OK, MURE_E_INVALID, MURE_E_STATE, MURE_E_NOMEM, MURE_E_DEVICE,
                      MURE_E_UNSUPPORTED, OP_GAUSS_FUZZ, OP_EFFECT_BLOCK, OP_ACT_INVERSE,
                      OP_NEURON_SWITCH, OP_WEIGHT_SHUFFLE)

__all__ = ["Mure", "MureError", "load_library", "LIB_PATH", "EXPORTED", "MURE_OK",
           "MURE_E_INVALID", "MURE_E_STATE", "MURE_E_NOMEM", "MURE_E_DEVICE",
           "MURE_E_UNSUPPORTED", "OP_GAUSS_FUZZ", "OP_EFFECT_BLOCK", "OP_ACT_INVERSE",
           "OP_NEURON_SWITCH", "OP_WEIGHT_SHUFFLE"]
