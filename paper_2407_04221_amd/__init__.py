"""MI355X-native batched Autoverse environment step (arXiv 2407.04221, Sec. 2.1).

Python binding of libautoverse.so (C ABI: include/autoverse.h).  The functions below carry
the C names and only marshal arguments: host numpy arrays for rules and checkpoints, torch
device tensors (device memory and streams) for maps, actions, rewards and done flags.
Every step runs in the library's HIP kernels; there is no CPU path.

`Batch` bundles one batch handle with its own output tensors for convenience.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libautoverse.so")

AV_OK, AV_EINVAL, AV_ENOMEM, AV_EDEVICE, AV_ESTATE = 0, 1, 2, 3, 4
AV_ENGINE_AUTO, AV_ENGINE_GENERIC, AV_ENGINE_LANE16, AV_ENGINE_WAVE, AV_ENGINE_ROWS = 0, 1, 2, 3, 4
AV_ENGINE_GROUP = 5
ENGINES = {"auto": AV_ENGINE_AUTO, "generic": AV_ENGINE_GENERIC, "lane16": AV_ENGINE_LANE16,
           "wave": AV_ENGINE_WAVE, "rows": AV_ENGINE_ROWS, "group": AV_ENGINE_GROUP}
ENGINE_NAMES = {v: k for k, v in ENGINES.items()}
AV_RULES_PARALLEL, AV_RULES_SEQUENTIAL = 0, 1
RULE_MODES = {"parallel": AV_RULES_PARALLEL, "sequential": AV_RULES_SEQUENTIAL}
AV_SITES_ROW_MAJOR, AV_SITES_RANDOM = 0, 1
SITE_ORDERS = {"rowmajor": AV_SITES_ROW_MAJOR, "random": AV_SITES_RANDOM}

# Every symbol include/autoverse.h declares.
ABI_SYMBOLS = ("av_create_batch", "av_load_rules", "av_set_rule_control", "av_reset",
               "av_step", "av_step_n", "av_step_observe",
               "av_get_maps", "av_observe", "av_rule_features", "av_state_ptr", "av_get_info",
               "av_get_state", "av_set_state", "av_set_stream", "av_destroy_batch",
               "av_mutate_maps", "av_mutate_rules", "av_search_create", "av_search_load_rules",
               "av_search_begin", "av_search_expand", "av_search_frontier", "av_search_destroy",
               "av_step_n_static", "av_last_error")


class av_config(ctypes.Structure):
    _fields_ = [("num_envs", ctypes.c_int32), ("height", ctypes.c_int32),
                ("width", ctypes.c_int32), ("channels", ctypes.c_int32),
                ("max_rules", ctypes.c_int32), ("max_pat_h", ctypes.c_int32),
                ("max_pat_w", ctypes.c_int32), ("per_env_rules", ctypes.c_int32),
                ("max_episode_steps", ctypes.c_int32), ("device", ctypes.c_int32),
                ("engine", ctypes.c_int32), ("rule_mode", ctypes.c_int32),
                ("stream", ctypes.c_void_p)]


class av_mutation(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("generation", ctypes.c_uint64),
                ("map_flip_p32", ctypes.c_uint32), ("map_channels", ctypes.c_uint32),
                ("entry_p32", ctypes.c_uint32), ("entry_channels", ctypes.c_uint32),
                ("reward_p32", ctypes.c_uint32), ("reward_lo", ctypes.c_int32),
                ("reward_hi", ctypes.c_int32)]


def p32(p: float) -> int:
    """Probability -> 32-bit threshold (an event happens iff its random word is below it)."""
    return max(0, min(0xFFFFFFFF, int(round(p * 2**32))))


def mutation(seed=0, generation=0, map_flip=0.0, map_channels=0xFFFFFFFF, entry=0.0,
             entry_channels=0xFFFFFFFF, reward=0.0, reward_lo=-1, reward_hi=1) -> av_mutation:
    m = av_mutation()
    m.seed, m.generation = seed, generation
    m.map_flip_p32, m.map_channels = p32(map_flip), map_channels
    m.entry_p32, m.entry_channels = p32(entry), entry_channels
    m.reward_p32, m.reward_lo, m.reward_hi = p32(reward), reward_lo, reward_hi
    return m


class av_search_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "height", "width", "channels", "max_rules", "max_pat_h", "max_pat_w",
        "max_episode_steps", "num_actions", "max_frontier", "table_log2", "device", "engine",
        "rule_mode", "best_first_k", "max_nodes", "hash_bits")] + [("stream", ctypes.c_void_p)]


class av_search_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in (
        "level", "parents", "children", "terminal", "survivors", "frontier", "visited",
        "best_visit")] + [("best_reward", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class av_info(ctypes.Structure):
    _fields_ = [("num_envs", ctypes.c_int32), ("height", ctypes.c_int32),
                ("width", ctypes.c_int32), ("channels", ctypes.c_int32),
                ("row_bytes", ctypes.c_int32), ("engine", ctypes.c_int32),
                ("state_bytes", ctypes.c_size_t), ("blob_bytes", ctypes.c_size_t)]


class AvError(RuntimeError):
    def __init__(self, fn: str, status: int, message: str):
        super().__init__(f"{fn}: status {status}: {message}")
        self.status = status
        self.message = message


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libautoverse.so; raise if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() or "
                           f"python paper_2407_04221_amd/build.py")
    lib = ctypes.CDLL(path)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sig = {
        "av_create_batch": ([ctypes.POINTER(av_config), ctypes.POINTER(P)], ctypes.c_int),
        "av_load_rules": ([P, I32, P, P, P, P], ctypes.c_int),
        "av_set_rule_control": ([P, P, P, I32, ctypes.c_uint64], ctypes.c_int),
        "av_reset": ([P, P], ctypes.c_int),
        "av_step": ([P, P, P, P], ctypes.c_int),
        "av_step_n": ([P, I32, P, P, P], ctypes.c_int),
        "av_step_observe": ([P, I32, P, P, P, I32, P], ctypes.c_int),
        "av_get_maps": ([P, P], ctypes.c_int),
        "av_observe": ([P, I32, P], ctypes.c_int),
        "av_rule_features": ([P, P], ctypes.c_int),
        "av_state_ptr": ([P], P),
        "av_get_info": ([P, ctypes.POINTER(av_info)], ctypes.c_int),
        "av_get_state": ([P, P, ctypes.POINTER(SZ)], ctypes.c_int),
        "av_set_state": ([P, P, SZ], ctypes.c_int),
        "av_set_stream": ([P, P], ctypes.c_int),
        "av_destroy_batch": ([P], ctypes.c_int),
        "av_mutate_maps": ([P, P, I32, I32, I32, I32, ctypes.POINTER(av_mutation), I32, P],
                           ctypes.c_int),
        "av_mutate_rules": ([I32, I32, I32, I32, I32, P, P, P, P, P, P, P,
                             ctypes.POINTER(av_mutation), I32, P], ctypes.c_int),
        "av_search_create": ([ctypes.POINTER(av_search_config), ctypes.POINTER(P)], ctypes.c_int),
        "av_search_load_rules": ([P, I32, P, P, P, P], ctypes.c_int),
        "av_search_begin": ([P, P], ctypes.c_int),
        "av_search_expand": ([P, ctypes.c_int64, ctypes.POINTER(av_search_info)], ctypes.c_int),
        "av_search_frontier": ([P, P, P, P], ctypes.c_int),
        "av_search_destroy": ([P], ctypes.c_int),
        "av_step_n_static": ([ctypes.POINTER(av_config), I32, P, P, P, P, P, P, P, I32, P, P, P],
                             ctypes.c_int),
        "av_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def av_last_error() -> str:
    return load_library().av_last_error().decode()


def _check(fn: str, rc: int):
    if rc != AV_OK:
        raise AvError(fn, rc, av_last_error())


def _torch():
    import torch
    return torch


def _dev_ptr(t, dtype, shape, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _host(a, dtype, name):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def current_stream_handle():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def av_create_batch(num_envs, height, width, channels, max_rules, max_pat_h, max_pat_w,
                    per_env_rules=False, max_episode_steps=0, device=None, engine="auto",
                    stream=None, rule_mode="parallel"):
    """Returns an opaque handle (ctypes.c_void_p).  stream: a torch.cuda.Stream, a raw
    handle, or None for torch's current stream on `device`."""
    torch = _torch()
    if device is None:
        device = torch.cuda.current_device()
    if stream is None:
        with torch.cuda.device(device):
            stream = current_stream_handle()
    elif hasattr(stream, "cuda_stream"):
        stream = ctypes.c_void_p(stream.cuda_stream)
    cfg = av_config(num_envs, height, width, channels, max_rules, max_pat_h, max_pat_w,
                    int(bool(per_env_rules)), max_episode_steps, int(device),
                    ENGINES[engine] if isinstance(engine, str) else int(engine),
                    RULE_MODES[rule_mode] if isinstance(rule_mode, str) else int(rule_mode),
                    stream)
    h = ctypes.c_void_p()
    _check("av_create_batch", load_library().av_create_batch(ctypes.byref(cfg), ctypes.byref(h)))
    return h


def av_load_rules(batch, shape, in_pat, out_pat, reward):
    """Host arrays: shape int32 [S][R][2], in_pat / out_pat int8 [S][R][C+1][mh][mw],
    reward int32 [S][R]."""
    shape, ps = _host(shape, np.int32, "shape")
    in_pat, pi = _host(in_pat, np.int8, "in_pat")
    out_pat, po = _host(out_pat, np.int8, "out_pat")
    reward, pr = _host(reward, np.int32, "reward")
    R = shape.shape[1] if shape.ndim == 3 else 0
    _check("av_load_rules", load_library().av_load_rules(batch, R, ps, pi, po, pr))


def av_set_rule_control(batch, limit=None, inhibit=None, order=AV_SITES_ROW_MAJOR, seed=0):
    """Host arrays or None: limit int32 [S][R] (0 = every match), inhibit uint8 [S][R][R]
    ([q][r]: q inhibits r, q < r); order AV_SITES_ROW_MAJOR / AV_SITES_RANDOM or its name."""
    pl = pi = None
    if limit is not None:
        limit, pl = _host(limit, np.int32, "limit")
    if inhibit is not None:
        inhibit, pi = _host(inhibit, np.uint8, "inhibit")
    order = SITE_ORDERS.get(order, order) if isinstance(order, str) else order
    _check("av_set_rule_control",
           load_library().av_set_rule_control(batch, pl, pi, int(order), int(seed)))


def av_mutate_maps(src, dst, m: av_mutation):
    """src, dst: device uint8 tensors [n][C][H][W] (may be the same tensor); runs on the
    current stream of their device."""
    torch = _torch()
    shp = tuple(src.shape)
    if len(shp) != 4:
        raise ValueError("maps must be [n][C][H][W]")
    n, C, H, W = shp
    ps = _dev_ptr(src, torch.uint8, shp, "src")
    pd = _dev_ptr(dst, torch.uint8, shp, "dst")
    _check("av_mutate_maps",
           load_library().av_mutate_maps(ps, pd, n, C, H, W, ctypes.byref(m), src.device.index,
                                         current_stream_handle()))


def av_mutate_rules(shape, in_src, out_src, reward_src, in_dst, out_dst, reward_dst,
                    m: av_mutation):
    """Device tensors in the av_load_rules layout: shape int32 [S][R][2], patterns int8
    [S][R][C+1][mh][mw], rewards int32 [S][R]; destinations may be the sources."""
    torch = _torch()
    S, R, C1, mh, mw = tuple(in_src.shape)
    args = [_dev_ptr(shape, torch.int32, (S, R, 2), "shape"),
            _dev_ptr(in_src, torch.int8, (S, R, C1, mh, mw), "in_src"),
            _dev_ptr(out_src, torch.int8, (S, R, C1, mh, mw), "out_src"),
            _dev_ptr(reward_src, torch.int32, (S, R), "reward_src"),
            _dev_ptr(in_dst, torch.int8, (S, R, C1, mh, mw), "in_dst"),
            _dev_ptr(out_dst, torch.int8, (S, R, C1, mh, mw), "out_dst"),
            _dev_ptr(reward_dst, torch.int32, (S, R), "reward_dst")]
    _check("av_mutate_rules",
           load_library().av_mutate_rules(S, R, C1 - 1, mh, mw, *args, ctypes.byref(m),
                                          in_src.device.index, current_stream_handle()))


def av_reset(batch, init_maps):
    info = av_get_info(batch)
    shp = (info["num_envs"], info["channels"], info["height"], info["width"])
    torch = _torch()
    _check("av_reset", load_library().av_reset(batch, _dev_ptr(init_maps, torch.uint8, shp,
                                                                 "init_maps")))


def av_step(batch, actions, rewards, done):
    torch = _torch()
    B = actions.shape[0] if hasattr(actions, "shape") else 0
    _check("av_step", load_library().av_step(
        batch, _dev_ptr(actions, torch.uint8, (B,), "actions"),
        _dev_ptr(rewards, torch.float32, (B,), "rewards"),
        _dev_ptr(done, torch.uint8, (B,), "done")))


def av_step_n(batch, k, actions, rewards, done):
    torch = _torch()
    B = actions.shape[1] if hasattr(actions, "shape") and actions.dim() == 2 else 0
    _check("av_step_n", load_library().av_step_n(
        batch, int(k), _dev_ptr(actions, torch.uint8, (k, B), "actions"),
        _dev_ptr(rewards, torch.float32, (k, B), "rewards"),
        _dev_ptr(done, torch.uint8, (k, B), "done")))


def av_step_n_static(num_envs, height, width, channels, max_rules, max_pat_h, max_pat_w,
                     rules, state, init, counters, actions, rewards, done, per_env_rules=False,
                     max_episode_steps=0, engine="auto", rule_mode="parallel", device=None,
                     stream=None):
    """k steps of caller-owned environments without device allocation.  rules: host
    (shape, in_pat, out_pat, reward) as av_load_rules; state / init: device uint8 tensors of
    the packed layout (C * B * H * row_bytes bytes); counters: device int32 [B]; actions
    uint8 [k][B], rewards float32 [k][B], done uint8 [k][B] device tensors."""
    torch = _torch()
    if device is None:
        device = torch.cuda.current_device()
    if stream is None:
        with torch.cuda.device(device):
            stream = current_stream_handle()
    elif hasattr(stream, "cuda_stream"):
        stream = ctypes.c_void_p(stream.cuda_stream)
    cfg = av_config(num_envs, height, width, channels, max_rules, max_pat_h, max_pat_w,
                    int(bool(per_env_rules)), max_episode_steps, int(device),
                    ENGINES[engine] if isinstance(engine, str) else int(engine),
                    RULE_MODES[rule_mode] if isinstance(rule_mode, str) else int(rule_mode),
                    stream)
    shape, ps = _host(rules[0], np.int32, "shape")
    in_pat, pi = _host(rules[1], np.int8, "in_pat")
    out_pat, po = _host(rules[2], np.int8, "out_pat")
    reward, pr = _host(rules[3], np.int32, "reward")
    R = shape.shape[1] if shape.ndim == 3 else 0
    k = actions.shape[0]
    row_bytes = 2 if width <= 16 else (4 if width <= 32 else 8)
    nbytes = channels * num_envs * height * row_bytes
    _check("av_step_n_static", load_library().av_step_n_static(
        ctypes.byref(cfg), R, ps, pi, po, pr,
        _dev_ptr(state, torch.uint8, (nbytes,), "state"),
        _dev_ptr(init, torch.uint8, (nbytes,), "init"),
        _dev_ptr(counters, torch.int32, (num_envs,), "counters"), int(k),
        _dev_ptr(actions, torch.uint8, (k, num_envs), "actions"),
        _dev_ptr(rewards, torch.float32, (k, num_envs), "rewards"),
        _dev_ptr(done, torch.uint8, (k, num_envs), "done")))


def av_step_observe(batch, k, actions, rewards, done, w, obs):
    """actions [k][B] uint8, rewards [k][B] float32, done [k][B] uint8, obs [B][C][w][w]
    uint8, all device tensors."""
    torch = _torch()
    info = av_get_info(batch)
    B, C = info["num_envs"], info["channels"]
    pa = _dev_ptr(actions, torch.uint8, (k, B), "actions")
    pr = _dev_ptr(rewards, torch.float32, (k, B), "rewards")
    pd = _dev_ptr(done, torch.uint8, (k, B), "done")
    po = _dev_ptr(obs, torch.uint8, (B, C, w, w), "obs")
    _check("av_step_observe", load_library().av_step_observe(batch, k, pa, pr, pd, w, po))


def av_get_maps(batch, dst):
    info = av_get_info(batch)
    shp = (info["num_envs"], info["channels"], info["height"], info["width"])
    torch = _torch()
    _check("av_get_maps", load_library().av_get_maps(batch, _dev_ptr(dst, torch.uint8, shp, "dst")))


def av_observe(batch, w, dst):
    """dst: device uint8 tensor [B][C][w][w]."""
    info = av_get_info(batch)
    shp = (info["num_envs"], info["channels"], w, w)
    torch = _torch()
    _check("av_observe", load_library().av_observe(batch, int(w),
                                                   _dev_ptr(dst, torch.uint8, shp, "dst")))


def av_rule_features(batch, dst):
    """dst: device uint8 tensor [S][R][2][2][C+1][max_pat_h][max_pat_w] (contiguous)."""
    torch = _torch()
    if not isinstance(dst, torch.Tensor) or not dst.is_cuda or dst.dtype != torch.uint8 \
            or not dst.is_contiguous():
        raise TypeError("dst must be a contiguous uint8 device tensor")
    _check("av_rule_features", load_library().av_rule_features(batch, ctypes.c_void_p(dst.data_ptr())))


def av_state_ptr(batch) -> int:
    p = load_library().av_state_ptr(batch)
    if not p:
        raise AvError("av_state_ptr", AV_EINVAL, av_last_error())
    return int(p)


def av_get_info(batch) -> dict:
    info = av_info()
    _check("av_get_info", load_library().av_get_info(batch, ctypes.byref(info)))
    return {f: getattr(info, f) for f, _ in av_info._fields_}


def av_get_state(batch) -> bytes:
    lib = load_library()
    n = ctypes.c_size_t(0)
    _check("av_get_state", lib.av_get_state(batch, None, ctypes.byref(n)))
    buf = ctypes.create_string_buffer(n.value)
    _check("av_get_state", lib.av_get_state(batch, buf, ctypes.byref(n)))
    return buf.raw[:n.value]


def av_set_state(batch, blob: bytes):
    buf = ctypes.create_string_buffer(blob, len(blob))
    _check("av_set_state", load_library().av_set_state(batch, buf, len(blob)))


def av_set_stream(batch, stream):
    if hasattr(stream, "cuda_stream"):
        stream = ctypes.c_void_p(stream.cuda_stream)
    _check("av_set_stream", load_library().av_set_stream(batch, stream))


def av_destroy_batch(batch):
    _check("av_destroy_batch", load_library().av_destroy_batch(batch))


class Batch:
    """A batch of B environments on one GPU, with reusable device buffers for actions,
    rewards and done flags."""

    def __init__(self, num_envs, height, width, channels, max_rules, max_pat_h, max_pat_w,
                 per_env_rules=False, max_episode_steps=0, device=None, engine="auto",
                 rule_mode="parallel"):
        torch = _torch()
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None
                                   else device)
        self.B, self.H, self.W, self.C = num_envs, height, width, channels
        self.h = av_create_batch(num_envs, height, width, channels, max_rules, max_pat_h,
                                 max_pat_w, per_env_rules, max_episode_steps,
                                 self.device.index, engine, rule_mode=rule_mode)
        self.rewards = torch.zeros(num_envs, dtype=torch.float32, device=self.device)
        self.done = torch.zeros(num_envs, dtype=torch.uint8, device=self.device)

    @classmethod
    def for_workload(cls, wl, B=None, device=None, engine="auto", rule_mode="parallel"):
        return cls(wl.B if B is None else B, wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w,
                   wl.per_env, wl.L, device=device, engine=engine, rule_mode=rule_mode)

    @property
    def info(self):
        return av_get_info(self.h)

    def load_rules(self, shape, in_pat, out_pat, reward):
        av_load_rules(self.h, shape, in_pat, out_pat, reward)
        self.S, self.R = (np.shape(shape)[0], np.shape(shape)[1]) if np.ndim(shape) == 3 \
            else (1, 0)

    def set_rule_control(self, limit=None, inhibit=None, order="rowmajor", seed=0):
        S, R = getattr(self, "S", 1), getattr(self, "R", 0)
        if limit is not None and np.shape(limit) != (S, R):
            raise ValueError(f"limit must have shape {(S, R)}, got {np.shape(limit)}")
        if inhibit is not None and np.shape(inhibit) != (S, R, R):
            raise ValueError(f"inhibit must have shape {(S, R, R)}, got {np.shape(inhibit)}")
        av_set_rule_control(self.h, limit, inhibit, order, seed)

    def reset(self, init_maps):
        torch = _torch()
        if not isinstance(init_maps, torch.Tensor):
            init_maps = torch.from_numpy(np.ascontiguousarray(init_maps, dtype=np.uint8))
        av_reset(self.h, init_maps.to(self.device).contiguous())

    def step(self, actions):
        """actions: uint8 device tensor [B]; returns this batch's (rewards, done) tensors."""
        av_step(self.h, actions, self.rewards, self.done)
        return self.rewards, self.done

    def step_n(self, actions, rewards=None, done=None):
        """actions [k][B] uint8 on the device; returns rewards [k][B], done [k][B]."""
        torch = _torch()
        k = actions.shape[0]
        if rewards is None:
            rewards = torch.empty((k, self.B), dtype=torch.float32, device=self.device)
        if done is None:
            done = torch.empty((k, self.B), dtype=torch.uint8, device=self.device)
        av_step_n(self.h, k, actions, rewards, done)
        return rewards, done

    def step_observe(self, actions, w, obs=None, rewards=None, done=None):
        """actions [k][B] on the device; returns (rewards [k][B], done [k][B], obs [B][C][w][w])
        with obs taken after the k-th step."""
        torch = _torch()
        k = actions.shape[0]
        if rewards is None:
            rewards = torch.empty((k, self.B), dtype=torch.float32, device=self.device)
        if done is None:
            done = torch.empty((k, self.B), dtype=torch.uint8, device=self.device)
        if obs is None:
            obs = torch.empty((self.B, self.C, w, w), dtype=torch.uint8, device=self.device)
        av_step_observe(self.h, k, actions, rewards, done, w, obs)
        return rewards, done, obs

    def maps(self, out=None):
        torch = _torch()
        if out is None:
            out = torch.empty((self.B, self.C, self.H, self.W), dtype=torch.uint8,
                              device=self.device)
        av_get_maps(self.h, out)
        return out

    def observe(self, w, out=None):
        torch = _torch()
        if out is None:
            out = torch.empty((self.B, self.C, w, w), dtype=torch.uint8, device=self.device)
        av_observe(self.h, w, out)
        return out

    def state_ptr(self) -> int:
        return av_state_ptr(self.h)

    def get_state(self) -> bytes:
        return av_get_state(self.h)

    def set_state(self, blob: bytes):
        av_set_state(self.h, blob)

    def close(self):
        if getattr(self, "h", None) is not None:
            av_destroy_batch(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Search:
    """Level-synchronous search over action sequences on one GPU (av_search_*): every level
    steps all (frontier node, action) pairs as one batch and deduplicates states in a device
    hash table.  The methods marshal arguments only."""

    def __init__(self, height, width, channels, max_rules, max_pat_h, max_pat_w,
                 max_episode_steps=0, num_actions=5, max_frontier=1 << 16, table_log2=20,
                 device=None, engine="auto", rule_mode="parallel", best_first_k=0,
                 max_nodes=1 << 20, hash_bits=0):
        torch = _torch()
        self.device = torch.device("cuda", torch.cuda.current_device() if device is None
                                   else device)
        self.H, self.W, self.C = height, width, channels
        cfg = av_search_config(height, width, channels, max_rules, max_pat_h, max_pat_w,
                               max_episode_steps, num_actions, max_frontier, table_log2,
                               self.device.index, ENGINES[engine] if isinstance(engine, str)
                               else engine, RULE_MODES[rule_mode] if isinstance(rule_mode, str)
                               else rule_mode, best_first_k, max_nodes, hash_bits,
                               current_stream_handle())
        h = ctypes.c_void_p()
        _check("av_search_create", load_library().av_search_create(ctypes.byref(cfg),
                                                                   ctypes.byref(h)))
        self.h = h
        self.n_front = 0

    def load_rules(self, shape, in_pat, out_pat, reward):
        shape, ps = _host(shape, np.int32, "shape")
        in_pat, pi = _host(in_pat, np.int8, "in_pat")
        out_pat, po = _host(out_pat, np.int8, "out_pat")
        reward, pr = _host(reward, np.int32, "reward")
        if shape.ndim == 3 and shape.shape[0] != 1:
            raise ValueError("a search takes one rule set (S = 1)")
        R = shape.shape[1] if shape.ndim == 3 else 0
        _check("av_search_load_rules",
               load_library().av_search_load_rules(self.h, R, ps, pi, po, pr))

    def begin(self, root):
        torch = _torch()
        if not isinstance(root, torch.Tensor):
            root = torch.from_numpy(np.ascontiguousarray(root, dtype=np.uint8))
        root = root.to(self.device).contiguous()
        p = _dev_ptr(root, torch.uint8, (self.C, self.H, self.W), "root")
        _check("av_search_begin", load_library().av_search_begin(self.h, p))
        self.n_front = 1

    def expand(self, max_children) -> dict:
        info = av_search_info()
        _check("av_search_expand",
               load_library().av_search_expand(self.h, int(max_children), ctypes.byref(info)))
        self.n_front = info.frontier
        return {k: getattr(info, k) for k, _ in av_search_info._fields_ if k != "reserved"}

    def frontier(self):
        """(maps uint8 [N][C][H][W], reward int32 [N], depth int32 [N]) device tensors."""
        torch = _torch()
        n = self.n_front
        maps = torch.empty((n, self.C, self.H, self.W), dtype=torch.uint8, device=self.device)
        reward = torch.empty(n, dtype=torch.int32, device=self.device)
        depth = torch.empty(n, dtype=torch.int32, device=self.device)
        if n:
            _check("av_search_frontier", load_library().av_search_frontier(
                self.h, ctypes.c_void_p(maps.data_ptr()), ctypes.c_void_p(reward.data_ptr()),
                ctypes.c_void_p(depth.data_ptr())))
        return maps, reward, depth

    def run(self, root, budget, max_levels=1 << 30):
        self.begin(root)
        out = []
        visited = 0
        while self.n_front and visited < budget and len(out) < max_levels:
            info = self.expand(budget - visited)
            visited = info["visited"]
            out.append(info)
        return out

    def close(self):
        if getattr(self, "h", None) is not None:
            load_library().av_search_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
