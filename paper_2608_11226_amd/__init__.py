"""Python binding of librollout, the MI355X GRPO rollout library.

Argument marshalling only: every step of the rollout runs in the library's
HIP kernels.  The functions below carry the names of the C ABI in
``include/rollout.h`` and take device pointers as integers (or torch tensors,
whose ``data_ptr()`` is passed); PyTorch is used by ``Engine`` only to
allocate device memory and to provide the stream.

The library must have been built (``python paper_2608_11226_amd/build.py``);
importing this package fails loudly when it has not.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# ROLLOUT_LIBRARY may name another build of the same library (the host-sanitizer build of build.py --sanitize)
LIB_PATH = os.environ.get("ROLLOUT_LIBRARY") or os.path.join(_PKG, "librollout.so")

OK, EINVAL, ENOMEM, EDEVICE, ESTATE, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
DTYPE_FP32, DTYPE_BF16, DTYPE_INT4 = 0, 1, 2
_NAMES = {EINVAL: "EINVAL", ENOMEM: "ENOMEM", EDEVICE: "EDEVICE", ESTATE: "ESTATE", EUNSUPPORTED: "EUNSUPPORTED"}

EXPORTED = (
    "rollout_plan", "rollout_init", "rollout_prefill", "rollout_decode_step", "rollout_sample",
    "grpo_advantages", "rollout_generate", "rollout_sync", "rollout_destroy", "rollout_last_error",
    "rollout_export_weight", "rollout_profile_decode_step", "rollout_generate_eos", "rollout_length_rewards",
    "rollout_sample_noalloc", "rollout_profile_projections",
)
NOALLOC_SCRATCH_BYTES = 64 << 20  # ROLLOUT_SAMPLE_NOALLOC_SCRATCH_BYTES
# include/occupancy.h: power metrics and threshold policy of the occupancy controller (host code)
EXPORTED_OCC = (
    "occ_rolling_mean", "occ_violation", "occ_normalize_budget", "occ_hysteresis_step", "occ_monitor_create",
    "occ_monitor_push", "occ_monitor_read", "occ_monitor_state", "occ_monitor_destroy",
)


class RolloutError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code


class ModelConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
        ("dtype", ctypes.c_int32), ("weight_seed", ctypes.c_uint64), ("weight_std", ctypes.c_double),
        ("kv_block_size", ctypes.c_int32), ("max_prompt_len", ctypes.c_int32),
        ("max_new_tokens", ctypes.c_int32), ("max_seqs_in_flight", ctypes.c_int32),
        ("hbm_budget_bytes", ctypes.c_uint64),
    ]


class Plan(ctypes.Structure):
    _fields_ = [
        ("seqs_in_flight_max", ctypes.c_int32), ("kv_blocks", ctypes.c_int32), ("arena_bytes", ctypes.c_uint64),
        ("weight_bytes", ctypes.c_uint64), ("kv_block_bytes", ctypes.c_uint64), ("kv_bytes", ctypes.c_uint64),
        ("work_bytes", ctypes.c_uint64),
    ]


class OccReading(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64), ("p_now_w", ctypes.c_double), ("p_5s_ago_w", ctypes.c_double),
        ("p10_w", ctypes.c_double), ("p30_w", ctypes.c_double), ("violation_rate", ctypes.c_double),
        ("excess_ws", ctypes.c_double), ("peak30_w", ctypes.c_double),
    ]


class ProjectionProfile(ctypes.Structure):
    _fields_ = [
        ("launches", ctypes.c_int32), ("avg_us", ctypes.c_double), ("bytes_per_launch", ctypes.c_double),
        ("flops_per_launch", ctypes.c_double),
    ]


class StepProfile(ctypes.Structure):
    _fields_ = [
        ("ms", ctypes.c_double * 3), ("launches", ctypes.c_int32 * 3),
        ("bytes", ctypes.c_double * 3), ("flops", ctypes.c_double * 3),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2608_11226_amd/build.py`")
    # torch's libraries link the HIP runtime it ships under an unversioned name;
    # loading torch first lets librollout's libamdhip64.so.7 / libhsa-runtime64.so.1
    # resolve to those same copies, so the process holds one HIP runtime.
    import torch  # noqa: F401

    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, f32, u64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_uint64, ctypes.c_double
    sig = {
        "rollout_plan": ([ctypes.POINTER(ModelConfig), i32, ctypes.POINTER(Plan)], i32),
        "rollout_init": ([ctypes.POINTER(ModelConfig), vp, u64, vp, ctypes.POINTER(vp)], i32),
        "rollout_prefill": ([vp, vp, i32, i32, i32, vp], i32),
        "rollout_decode_step": ([vp, vp, vp], i32),
        "rollout_sample": ([vp, vp, i32, f32, f32, vp, vp], i32),
        "grpo_advantages": ([vp, i32, i32, f32, i32, vp, vp, vp], i32),
        "rollout_generate": ([vp, vp, i32, i32, i32, i32, i32, f32, f32, vp, vp], i32),
        "rollout_sync": ([vp], i32),
        "rollout_destroy": ([vp], None),
        "rollout_last_error": ([vp], ctypes.c_char_p),
        "rollout_export_weight": ([vp, i32, vp], i32),
        "rollout_profile_decode_step": ([vp, vp, vp, ctypes.POINTER(StepProfile)], i32),
        "rollout_generate_eos": ([vp, vp, i32, i32, i32, i32, i32, f32, f32, vp, vp, i32, i32, i32, vp, vp, vp,
                                  ctypes.POINTER(i32)], i32),
        "rollout_length_rewards": ([vp, i32, i32, vp, vp, vp], i32),
        "rollout_sample_noalloc": ([vp, i32, i32, f32, f32, vp, vp, vp], i32),
        "rollout_profile_projections": ([vp, i32, vp, ctypes.POINTER(ProjectionProfile)], i32),
        "occ_rolling_mean": ([vp, ctypes.c_int64, f64, f64, vp], i32),
        "occ_violation": ([vp, ctypes.c_int64, f64, f64, ctypes.POINTER(f64), ctypes.POINTER(f64)], i32),
        "occ_normalize_budget": ([f64, f64, f64], f64),
        "occ_hysteresis_step": ([i32, i32, f64, f64, f64, f64, f64], i32),
        "occ_monitor_create": ([f64, f64], vp),
        "occ_monitor_push": ([vp, f64], i32),
        "occ_monitor_read": ([vp, ctypes.POINTER(OccReading)], i32),
        "occ_monitor_state": ([vp, i32, i32, f64, vp], i32),
        "occ_monitor_destroy": ([vp], None),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


lib = _load()


def _ptr(x) -> int | None:
    """Device pointer of a tensor (data_ptr) or an integer address; None stays NULL."""
    if x is None:
        return None
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    return int(x)


def _check(code: int, ctx=None):
    if code != OK:
        raise RolloutError(code, lib.rollout_last_error(ctx).decode())


# ---------------------------------------------------------------------------
# C ABI, one wrapper per entry point
# ---------------------------------------------------------------------------
def rollout_plan(cfg: ModelConfig, group_size: int) -> Plan:
    out = Plan()
    _check(lib.rollout_plan(ctypes.byref(cfg), group_size, ctypes.byref(out)))
    return out


def rollout_init(cfg: ModelConfig, arena, arena_bytes: int, stream=None) -> int:
    ctx = ctypes.c_void_p()
    _check(lib.rollout_init(ctypes.byref(cfg), _ptr(arena), arena_bytes, _ptr(stream), ctypes.byref(ctx)))
    return ctx.value


def rollout_prefill(ctx, prompts, n_prompts: int, prompt_len: int, group_size: int, logits):
    _check(lib.rollout_prefill(ctx, _ptr(prompts), n_prompts, prompt_len, group_size, _ptr(logits)), ctx)


def rollout_decode_step(ctx, tokens, logits):
    _check(lib.rollout_decode_step(ctx, _ptr(tokens), _ptr(logits)), ctx)


def rollout_sample(ctx, logits, n_seqs: int, temperature: float, top_p: float, uniforms, tokens_out):
    _check(lib.rollout_sample(ctx, _ptr(logits), n_seqs, temperature, top_p, _ptr(uniforms), _ptr(tokens_out)), ctx)


def rollout_sample_noalloc(logits, n_seqs: int, vocab: int, temperature: float, top_p: float, uniforms, tokens_out,
                           stream=None):
    _check(lib.rollout_sample_noalloc(_ptr(logits), n_seqs, vocab, temperature, top_p, _ptr(uniforms),
                                      _ptr(tokens_out), _ptr(stream)))


def grpo_advantages(rewards, n_groups: int, group_size: int, eps: float, std_ddof: int, adv, zero_var=None,
                    stream=None):
    _check(lib.grpo_advantages(_ptr(rewards), n_groups, group_size, eps, std_ddof, _ptr(adv), _ptr(zero_var),
                               _ptr(stream)))


def rollout_generate(ctx, prompts, n_prompts: int, prompt_len: int, group_size: int, seqs_in_flight: int,
                     max_new_tokens: int, temperature: float, top_p: float, uniforms, tokens_out):
    _check(lib.rollout_generate(ctx, _ptr(prompts), n_prompts, prompt_len, group_size, seqs_in_flight,
                                max_new_tokens, temperature, top_p, _ptr(uniforms), _ptr(tokens_out)), ctx)


def rollout_generate_eos(ctx, prompts, n_prompts: int, prompt_len: int, group_size: int, seqs_in_flight: int,
                         max_new_tokens: int, temperature: float, top_p: float, uniforms, stop_ids, n_stop: int,
                         refill_interval: int, whole_groups: int, tokens_out, lengths_out,
                         admit_step_out=None) -> int:
    """Returns the number of decode steps run."""
    steps = ctypes.c_int32(0)
    _check(lib.rollout_generate_eos(ctx, _ptr(prompts), n_prompts, prompt_len, group_size, seqs_in_flight,
                                    max_new_tokens, temperature, top_p, _ptr(uniforms), _ptr(stop_ids), n_stop,
                                    refill_interval, whole_groups, _ptr(tokens_out), _ptr(lengths_out),
                                    _ptr(admit_step_out), ctypes.byref(steps)), ctx)
    return steps.value


def rollout_length_rewards(lengths, n: int, target: int, rewards, total_tokens=None, stream=None):
    _check(lib.rollout_length_rewards(_ptr(lengths), n, target, _ptr(rewards), _ptr(total_tokens), _ptr(stream)))


def rollout_sync(ctx):
    _check(lib.rollout_sync(ctx), ctx)


def rollout_destroy(ctx):
    lib.rollout_destroy(ctx)


def rollout_last_error(ctx=None) -> str:
    return lib.rollout_last_error(ctx).decode()


def rollout_export_weight(ctx, tensor_id: int, out):
    _check(lib.rollout_export_weight(ctx, tensor_id, _ptr(out)), ctx)


def rollout_profile_projections(ctx, reps: int, logits) -> ProjectionProfile:
    out = ProjectionProfile()
    _check(lib.rollout_profile_projections(ctx, reps, _ptr(logits), ctypes.byref(out)), ctx)
    return out


def rollout_profile_decode_step(ctx, tokens, logits) -> StepProfile:
    out = StepProfile()
    _check(lib.rollout_profile_decode_step(ctx, _ptr(tokens), _ptr(logits), ctypes.byref(out)), ctx)
    return out


# ---------------------------------------------------------------------------
# Model shapes of the synthetic workloads
# ---------------------------------------------------------------------------
SHAPES = {
    # n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab, rope_theta
    "tiny": (2, 128, 4, 4, 32, 512, 1024, 1e4),
    "7b": (28, 3584, 28, 4, 128, 18944, 152064, 1e6),
    "14b": (48, 5120, 40, 8, 128, 13824, 152064, 1e6),
    "72b": (80, 8192, 64, 8, 128, 29568, 152064, 1e6),
}


# ---------------------------------------------------------------------------
# include/occupancy.h (host code: arrays are float64 NumPy arrays)
# ---------------------------------------------------------------------------
def _f64(a):
    import numpy as np

    return np.ascontiguousarray(a, dtype=np.float64)


def occ_rolling_mean(p, dt_s: float, window_s: float):
    import numpy as np

    p = _f64(p)
    out = np.empty_like(p)
    _check(lib.occ_rolling_mean(p.ctypes.data, len(p), dt_s, window_s, out.ctypes.data))
    return out


def occ_violation(p30, budget_w: float, dt_s: float):
    p30 = _f64(p30)
    rate, excess = ctypes.c_double(), ctypes.c_double()
    _check(lib.occ_violation(p30.ctypes.data, len(p30), budget_w, dt_s, ctypes.byref(rate), ctypes.byref(excess)))
    return rate.value, excess.value


def occ_normalize_budget(budget_cal_w: float, p4_new_w: float, p4_cal_w: float) -> float:
    return lib.occ_normalize_budget(budget_cal_w, p4_new_w, p4_cal_w)


def occ_hysteresis_step(level_idx: int, n_levels: int, p30_w: float, p10_w: float, drop_w: float, climb30_w: float,
                        climb10_w: float) -> int:
    r = lib.occ_hysteresis_step(level_idx, n_levels, p30_w, p10_w, drop_w, climb30_w, climb10_w)
    if r < 0:
        raise RolloutError(EINVAL, "level index outside [0, n_levels)")
    return r


class OccMonitor:
    """occ_monitor_*: eq. (1) means and eqs. (2)-(3) accumulated over pushed power samples."""

    def __init__(self, dt_s: float, budget_w: float):
        self.h = lib.occ_monitor_create(dt_s, budget_w)
        if not self.h:
            raise RolloutError(EINVAL, "occ_monitor_create: dt_s must be > 0")
        self.dt_s, self.budget_w = dt_s, budget_w

    def push(self, power_w: float):
        _check(lib.occ_monitor_push(self.h, power_w))

    def read(self) -> OccReading:
        r = OccReading()
        _check(lib.occ_monitor_read(self.h, ctypes.byref(r)))
        return r

    def state(self, level: int, prev_level: int, prev_duration_s: float):
        import numpy as np

        out = np.empty(8, dtype=np.float64)
        _check(lib.occ_monitor_state(self.h, level, prev_level, prev_duration_s, out.ctypes.data))
        return out

    def close(self):
        if self.h:
            lib.occ_monitor_destroy(self.h)
            self.h = None

    def __del__(self):
        self.close()


def model_config(shape, dtype: int, max_prompt_len: int, max_new_tokens: int, max_seqs_in_flight: int,
                 n_layers: int | None = None, weight_seed: int = 0, weight_std: float = 0.02,
                 kv_block_size: int = 16, rms_eps: float = 1e-6, hbm_budget_bytes: int = 0) -> ModelConfig:
    """ModelConfig for a named shape (or a tuple in SHAPES order); n_layers overrides the depth."""
    t = SHAPES[shape] if isinstance(shape, str) else tuple(shape)
    return ModelConfig(
        n_layers=n_layers or t[0], d_model=t[1], n_heads=t[2], n_kv_heads=t[3], head_dim=t[4], d_ff=t[5],
        vocab=t[6], rms_eps=rms_eps, rope_theta=t[7], dtype=dtype, weight_seed=weight_seed,
        weight_std=weight_std, kv_block_size=kv_block_size, max_prompt_len=max_prompt_len,
        max_new_tokens=max_new_tokens, max_seqs_in_flight=max_seqs_in_flight,
        hbm_budget_bytes=hbm_budget_bytes)


class Engine:
    """A context plus the device arena it lives in (torch supplies memory and the stream)."""

    def __init__(self, cfg: ModelConfig, group_size: int = 1, device: str = "cuda:0", stream=None):
        import torch

        self.torch = torch
        self.device = torch.device(device)
        plan = rollout_plan(cfg, group_size)
        cfg.max_seqs_in_flight = plan.seqs_in_flight_max
        plan = rollout_plan(cfg, group_size)
        self.cfg, self.plan = cfg, plan
        self.arena = torch.empty(plan.arena_bytes, dtype=torch.uint8, device=self.device)
        self.stream = stream or torch.cuda.Stream(device=self.device)
        self.ctx = rollout_init(cfg, self.arena, plan.arena_bytes, self.stream.cuda_stream)

    @property
    def stream_handle(self) -> int:
        return self.stream.cuda_stream

    def synchronize(self):
        rollout_sync(self.ctx)

    def close(self):
        if self.ctx:
            rollout_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
