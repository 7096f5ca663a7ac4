"""MI355X (gfx950) experience-replay hot path: trajectory selection and
collection behind the C ABI in include/gear.h (GEAR, arXiv 2310.05205).

The HIP kernels and the C ABI are in ``csrc/`` and build into ``libgear.so``
(``python -m paper_2310_05205_amd.build``); ``gear`` is the ctypes binding.
"""
from .gear import (GEAR_DEVICE, GEAR_FIFO, GEAR_HOST_PINNED, GEAR_LIFO, GEAR_PRIORITIZED,  # noqa: F401
                   GEAR_STATUS_BAD_INDEX, GEAR_STATUS_NO_WEIGHT, GEAR_UNIFORM, GearError, Table)
