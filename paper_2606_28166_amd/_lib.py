"""ctypes binding of libtandem.so (the C ABI declared in include/tandem.h).

Argument marshalling only: every step of the tandem rollout runs in the HIP
kernels of the library.  Importing this module loads the library and raises
if it has not been built (python -m paper_2606_28166_amd.build).
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtandem.so")

OK, E_ARG, E_SHAPE, E_CAPACITY, E_STATE, E_HIP, E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
JUNIOR, SENIOR, DRAW = 0, 1, 2
REDRAW, SWITCH, ALTERNATE = 0, 1, 2
BF16, F32 = 0, 1


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("rope_theta", C.c_float), ("rms_eps", C.c_float),
                ("qk_norm", C.c_int32), ("weight_dtype", C.c_int32)]


class Model(C.Structure):
    _fields_ = [("cfg", ModelCfg), ("embed", C.c_void_p), ("layers", C.POINTER(C.c_void_p)),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)]


class SwitchCfg(C.Structure):
    _fields_ = [("mode", C.c_int32), ("p", C.c_double), ("cap_k", C.c_int32),
                ("boundary_bits", C.c_void_p), ("first_owner", C.c_int32)]


class SampleCfg(C.Structure):
    _fields_ = [("temperature", C.c_float), ("eos_id", C.c_int32), ("eos_bias_senior", C.c_float),
                ("eos_bias_junior", C.c_float), ("max_new_tokens", C.c_int32), ("seed", C.c_uint64)]


class Capacity(C.Structure):
    _fields_ = [("max_seqs", C.c_int32), ("max_ctx", C.c_int32), ("max_prefill_tokens", C.c_int32)]


class Outputs(C.Structure):
    _fields_ = [("tokens", C.c_void_p), ("owner", C.c_void_p), ("senior_logprob", C.c_void_p),
                ("length", C.c_void_p)]


class Debug(C.Structure):
    _fields_ = [("sampled", C.c_void_p), ("margin", C.c_void_p), ("logits_senior", C.c_void_p),
                ("logits_junior", C.c_void_p)]


class GrpoCfg(C.Structure):
    _fields_ = [("n_groups", C.c_int32), ("group_size", C.c_int32), ("max_new_tokens", C.c_int32),
                ("clip_eps", C.c_float)]


EXPORTS = ("tandem_workspace_size", "tandem_init", "tandem_prefill", "tandem_step",
           "tandem_step_forced", "tandem_score_step", "tandem_get_state", "tandem_timing_enable", "tandem_timing_read",
           "tandem_last_error", "tandem_status_string", "tandem_destroy", "tandem_grpo_workspace_size",
           "tandem_grpo_loss", "tandem_grpo_loss_noalloc")
K_ATTENTION, K_GEMM, K_SAMPLE, K_OTHER = 0, 1, 2, 3
TIMING_SERIAL = 1 << 8          # timing flag: run the two forwards one after the other
TIMING_EAGER = 1 << 9           # timing flag: launch every kernel from the host (no step graph)
TIMING_SEPARATE_SAMPLE = 1 << 10  # flag: store the logits and sample in a separate pass (no sampling in the LM heads)


def _load():
    # PyTorch-ROCm brings its own HIP/HSA runtime; load it first so that the
    # library's libamdhip64 dependency binds to that same instance.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_28166_amd.build`")
    lib = C.CDLL(LIB_PATH)
    P = C.c_void_p
    st = C.c_int
    lib.tandem_workspace_size.argtypes = [C.POINTER(ModelCfg), C.POINTER(ModelCfg), C.POINTER(Capacity),
                                          C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]
    lib.tandem_workspace_size.restype = st
    lib.tandem_init.argtypes = [C.POINTER(Model), C.POINTER(Model), C.POINTER(SwitchCfg), C.POINTER(SampleCfg),
                                C.POINTER(Capacity), P, C.c_size_t, P, C.c_size_t, C.POINTER(Outputs), P,
                                C.POINTER(P)]
    lib.tandem_init.restype = st
    lib.tandem_prefill.argtypes = [P, P, C.POINTER(C.c_int32), C.c_int32, C.c_int32]
    lib.tandem_prefill.restype = st
    lib.tandem_step.argtypes = [P, C.POINTER(C.c_int32)]
    lib.tandem_step.restype = st
    lib.tandem_step_forced.argtypes = [P, P, C.POINTER(Debug), C.POINTER(C.c_int32)]
    lib.tandem_step_forced.restype = st
    lib.tandem_score_step.argtypes = [P, P]
    lib.tandem_score_step.restype = st
    lib.tandem_get_state.argtypes = [P, P, P, P, P, P]
    lib.tandem_get_state.restype = st
    lib.tandem_timing_enable.argtypes = [P, C.c_int32]
    lib.tandem_timing_enable.restype = st
    lib.tandem_timing_read.argtypes = [P, C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]
    lib.tandem_timing_read.restype = st
    lib.tandem_last_error.argtypes = [P]
    lib.tandem_last_error.restype = C.c_char_p
    lib.tandem_status_string.argtypes = [C.c_int]
    lib.tandem_status_string.restype = C.c_char_p
    lib.tandem_destroy.argtypes = [P]
    lib.tandem_destroy.restype = None
    lib.tandem_grpo_workspace_size.argtypes = [C.POINTER(GrpoCfg), C.POINTER(C.c_size_t)]
    lib.tandem_grpo_workspace_size.restype = st
    lib.tandem_grpo_loss.argtypes = [C.POINTER(GrpoCfg), P, P, P, P, P, P, P, P, P, P, C.c_size_t, P]
    lib.tandem_grpo_loss.restype = st
    lib.tandem_grpo_loss_noalloc.argtypes = [C.POINTER(GrpoCfg), P, P, P, P, P, P, P, P, P, P]
    lib.tandem_grpo_loss_noalloc.restype = st
    return lib


lib = _load()


class TandemError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{lib.tandem_status_string(status).decode()}: {msg}")
        self.status = status


def check(status: int, handle=None) -> None:
    if status != OK:
        raise TandemError(status, lib.tandem_last_error(handle).decode())


# ------------------------------------------------- same-named thin wrappers

def _ref(x):
    return C.byref(x) if x is not None else None


def tandem_workspace_size(sen: ModelCfg, jun, cap: Capacity):
    """jun None: the senior alone."""
    kv, sc = C.c_size_t(), C.c_size_t()
    check(lib.tandem_workspace_size(C.byref(sen), _ref(jun), C.byref(cap), C.byref(kv), C.byref(sc)))
    return kv.value, sc.value


def tandem_init(sen: Model, jun, sw, smp: SampleCfg, cap: Capacity, kv_ptr: int,
                kv_bytes: int, scratch_ptr: int, scratch_bytes: int, out: Outputs, stream: int):
    """jun None: a single-model rollout of the senior (sw may be None)."""
    h = C.c_void_p()
    check(lib.tandem_init(C.byref(sen), _ref(jun), _ref(sw), C.byref(smp), C.byref(cap), kv_ptr,
                          kv_bytes, scratch_ptr, scratch_bytes, C.byref(out), stream, C.byref(h)))
    return h


def tandem_prefill(h, tokens_ptr: int, offsets, n_prompts: int, G: int) -> None:
    arr = (C.c_int32 * len(offsets))(*[int(x) for x in offsets])
    check(lib.tandem_prefill(h, tokens_ptr, arr, n_prompts, G), h)


def tandem_step(h, want_active: bool = False):
    n = C.c_int32(-1)
    check(lib.tandem_step(h, C.byref(n) if want_active else None), h)
    return n.value if want_active else None


def tandem_step_forced(h, forced_ptr: int, dbg: Debug = None, want_active: bool = False):
    n = C.c_int32(-1)
    check(lib.tandem_step_forced(h, forced_ptr, C.byref(dbg) if dbg is not None else None,
                                 C.byref(n) if want_active else None), h)
    return n.value if want_active else None


def tandem_score_step(h, scores_ptr: int) -> None:
    check(lib.tandem_score_step(h, scores_ptr), h)


def tandem_get_state(h, n_seq: int):
    arrs = [(C.c_int32 * n_seq)() for _ in range(5)]
    check(lib.tandem_get_state(h, *[C.cast(a, C.c_void_p) for a in arrs]), h)
    return [list(a) for a in arrs]


def tandem_timing_enable(h, class_mask: int) -> None:
    check(lib.tandem_timing_enable(h, int(class_mask)), h)


def tandem_timing_read(h, kernel_class: int):
    ms, n = C.c_double(), C.c_int64()
    check(lib.tandem_timing_read(h, kernel_class, C.byref(ms), C.byref(n)), h)
    return ms.value, n.value


def tandem_destroy(h) -> None:
    lib.tandem_destroy(h)


def tandem_grpo_workspace_size(cfg: GrpoCfg) -> int:
    n = C.c_size_t()
    check(lib.tandem_grpo_workspace_size(C.byref(cfg), C.byref(n)))
    return n.value


def tandem_grpo_loss(cfg: GrpoCfg, rewards: int, owner: int, length: int, logp_old: int, logp_new,
                     advantages: int, grad, loss: int, n_masked: int, workspace: int, workspace_bytes: int,
                     stream: int) -> None:
    check(lib.tandem_grpo_loss(C.byref(cfg), rewards, owner, length, logp_old, logp_new, advantages, grad,
                               loss, n_masked, workspace, workspace_bytes, stream))


def tandem_grpo_loss_noalloc(cfg: GrpoCfg, rewards: int, owner: int, length: int, logp_old: int, logp_new,
                             advantages: int, grad, loss: int, n_masked: int, stream: int) -> None:
    check(lib.tandem_grpo_loss_noalloc(C.byref(cfg), rewards, owner, length, logp_old, logp_new, advantages,
                                       grad, loss, n_masked, stream))
