"""ctypes view of libgrpo's C ABI (include/grpo.h).  Marshalling only."""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
SO = os.path.join(PKG, "libgrpo.so")

GRPO_OK = 0
GRPO_ERR_ARG = -1
GRPO_ERR_SHAPE = -2
GRPO_ERR_DTYPE = -3
GRPO_ERR_WORKSPACE = -4
GRPO_ERR_ALIGN = -5
GRPO_ERR_HIP = -6

GRPO_F32 = 0
GRPO_BF16 = 1
GRPO_NORM_TRAJ_STEPS = 0
GRPO_NORM_CONST_K = 1
GRPO_ADV_GROUP_NORM = 0
GRPO_ADV_SUCCESS_FILTER = 1

GRPO_NOALLOC_SCRATCH_BYTES = 24 << 20

GRPO_FLAG_ACTION = 1
GRPO_FLAG_OFFSETS = 2
GRPO_FLAG_NONFINITE = 4

P = ctypes.c_void_p


class Segments(ctypes.Structure):
    _fields_ = [("n_traj", ctypes.c_int32), ("group_size", ctypes.c_int32), ("n_steps", ctypes.c_int32),
                ("step_tok_off", P), ("traj_step_off", P)]


class LossParams(ctypes.Structure):
    _fields_ = [("norm", ctypes.c_int32), ("k", ctypes.c_float), ("eps_low", ctypes.c_float),
                ("eps_high", ctypes.c_float), ("dual_clip_c", ctypes.c_float), ("grad_scale", ctypes.c_float),
                ("n_groups_total", ctypes.c_double)]


class Aux(ctypes.Structure):
    _fields_ = [("token_logp", P), ("tok_traj", P), ("traj_tok_off", P), ("gather_idx", P), ("traj_loss", P),
                ("clip_counts", P), ("ratio_stats", P), ("error_flags", P), ("hot_begin", P), ("hot_end", P)]


class GrpoError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_str(status)} ({status})")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Loads the built library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(SO):
            raise RuntimeError(f"libgrpo.so not built at {SO}: run paper_2606_05597_amd/build.py")
        lib = ctypes.CDLL(SO)
        I32, I64, SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        lib.grpo_advantages.argtypes = [P, I32, I32, I32, ctypes.c_float, P, P]
        lib.grpo_advantages.restype = ctypes.c_int
        lib.grpo_advantages_ex.argtypes = [P, I32, I32, I32, I32, ctypes.c_float, P, P, P, P]
        lib.grpo_advantages_ex.restype = ctypes.c_int
        lib.grpo_loss_workspace_bytes.argtypes = [I64, I32]
        lib.grpo_loss_workspace_bytes.restype = SZ
        lib.grpo_loss_fwd_bwd.argtypes = [P, ctypes.c_int, I64, I64, I64, P, P, P, P,
                                          ctypes.POINTER(Segments), ctypes.POINTER(LossParams), P, P,
                                          ctypes.POINTER(Aux), P, SZ, P]
        lib.grpo_loss_fwd_bwd.restype = ctypes.c_int
        lib.grpo_loss_fwd_bwd_noalloc.argtypes = lib.grpo_loss_fwd_bwd.argtypes[:14] + [P]
        lib.grpo_loss_fwd_bwd_noalloc.restype = ctypes.c_int
        lib.fused_lmhead_workspace_bytes.argtypes = [I64, I64, I64, I32, I32]
        lib.fused_lmhead_workspace_bytes.restype = SZ
        lib.fused_lmhead_grpo.argtypes = [P, P, I64, I64, I64, I32, P, P, P, P, ctypes.POINTER(Segments),
                                          ctypes.POINTER(LossParams), P, P, P, I32, ctypes.POINTER(Aux), P, SZ, P]
        lib.fused_lmhead_grpo.restype = ctypes.c_int
        lib.fused_lmhead_blocked_workspace_bytes.argtypes = [I64, I64, I64, I32, I32]
        lib.fused_lmhead_blocked_workspace_bytes.restype = SZ
        lib.fused_lmhead_grpo_blocked.argtypes = lib.fused_lmhead_grpo.argtypes + [P]
        lib.fused_lmhead_grpo_blocked.restype = ctypes.c_int
        lib.fused_lmhead_token_logp_workspace_bytes.argtypes = [I64, I64, I64]
        lib.fused_lmhead_token_logp_workspace_bytes.restype = SZ
        lib.fused_lmhead_token_logp.argtypes = [P, P, I64, I64, I64, P, P, P, P, P, SZ, P]
        lib.fused_lmhead_token_logp.restype = ctypes.c_int
        lib.grpo_token_logp.argtypes = [P, ctypes.c_int, I64, I64, I64, P, P, P, P, P]
        lib.grpo_token_logp.restype = ctypes.c_int
        lib.grpo_vocab_shard_stats.argtypes = [P, ctypes.c_int, I64, I64, I64, I64, P, P, P, P]
        lib.grpo_vocab_shard_stats.restype = ctypes.c_int
        lib.grpo_loss_fwd_bwd_vocab_shard.argtypes = [P, ctypes.c_int, I64, I64, I64, I64, I64, P, I32, P, P, P, P,
                                                      ctypes.POINTER(Segments), ctypes.POINTER(LossParams), P, P,
                                                      ctypes.POINTER(Aux), P, SZ, P]
        lib.grpo_loss_fwd_bwd_vocab_shard.restype = ctypes.c_int
        lib.fused_lmhead_vocab_shard_stats_workspace_bytes.argtypes = [I64, I64, I64]
        lib.fused_lmhead_vocab_shard_stats_workspace_bytes.restype = SZ
        lib.fused_lmhead_vocab_shard_stats.argtypes = [P, P, I64, I64, I64, I64, P, P, P, P, SZ, P]
        lib.fused_lmhead_vocab_shard_stats.restype = ctypes.c_int
        lib.fused_lmhead_grpo_vocab_shard.argtypes = [P, P, I64, I64, I64, I64, I64, I32, P, I32, P, P, P, P,
                                                      ctypes.POINTER(Segments), ctypes.POINTER(LossParams), P, P, P,
                                                      I32, ctypes.POINTER(Aux), P, P, SZ, P]
        lib.fused_lmhead_vocab_shard_logits_bytes.argtypes = [I64, I64]
        lib.fused_lmhead_vocab_shard_logits_bytes.restype = SZ
        lib.fused_lmhead_grpo_vocab_shard.restype = ctypes.c_int
        lib.grpo_status_str.argtypes = [ctypes.c_int]
        lib.grpo_status_str.restype = ctypes.c_char_p
        _lib = lib
    return _lib


def status_str(status: int) -> str:
    return load().grpo_status_str(int(status)).decode()
