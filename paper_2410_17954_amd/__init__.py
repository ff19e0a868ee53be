"""MI355X-native MoE-layer hot path of ExpertFlow (arXiv 2410.17954).

The five steps -- gating, token scheduling, expert-major permutation, grouped
SwiGLU expert FFN and weighted combine -- run as HIP kernels for gfx950 inside
libmoeflow.so, a C-ABI library declared in include/moeflow.h. This package is
the thin Python binding over it (argument marshalling only); see `ops`.
Importing the package loads neither torch nor the library; the first call of an
operation does, and it raises if the library has not been built.
"""
_OPS = ("route", "schedule", "permute", "expert_ffn", "combine",
        "schedule_workspace", "permute_workspace", "expert_ffn_workspace",
        "plan_slots", "MoeError")

__all__ = list(_OPS)


def __getattr__(name):
    if name in _OPS:
        from . import ops
        return getattr(ops, name)
    raise AttributeError(name)
