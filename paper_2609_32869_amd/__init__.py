"""Whisper-Flash draft-and-verify step on MI355X (gfx950).

The step runs in the HIP kernels of ``libwf.so`` behind the C ABI of
``include/wf.h``; ``binding`` marshals arguments from Python.
"""
from .binding import (WhisperFlash, WhisperEncoder, WfError, load_library, make_config, make_encoder_config,
                      to_device_storage, rng_words_host, rng_words_device, EXPORTS, LIB_PATH)

__all__ = ["WhisperFlash", "WhisperEncoder", "WfError", "load_library", "make_config", "make_encoder_config",
           "to_device_storage", "rng_words_host", "rng_words_device", "EXPORTS", "LIB_PATH"]
