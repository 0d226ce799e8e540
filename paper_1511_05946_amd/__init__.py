"""MI355X (gfx950) ACDC / AFDF cascade library: HIP kernels behind a C ABI
(include/acdc.h) with a thin torch binding."""

from .acdc import (FLAG_COMPLEX, FLAG_PERM, FLAG_RELU, ACDCCascade, ACDCError, acdc_cascade,
                   backward, forward, prepare, supported)

__all__ = ["FLAG_PERM", "FLAG_RELU", "FLAG_COMPLEX", "forward", "backward", "prepare", "supported",
           "acdc_cascade", "ACDCCascade", "ACDCError"]
