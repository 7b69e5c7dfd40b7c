"""MI355X-native batched dynamic-routing executor (the hot path of DyCL,
arXiv 2307.04963): a C-ABI library of gfx950 kernels plus a thin binding."""

from .lowering import lower, lower_json  # noqa: F401
