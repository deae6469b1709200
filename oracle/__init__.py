"""ctypes wrapper of the CPU oracle (oracle/avo.c).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only the test-suite, the smoke check and
the benchmark's CPU-baseline leg import this package.  It never loads the GPU library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "avo.c")
LIB = os.path.join(HERE, "libavo.so")

AVO_OK, AVO_EINVAL, AVO_ENOMEM, AVO_ESTATE = 0, 1, 2, 4


def build(out: str = LIB, src: str = SRC, extra=()) -> str:
    """Compile the oracle with gcc (-O2, OpenMP); returns the library path."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-Wall", "-Wextra", "-shared", "-fPIC",
           *extra, src, "-o", out]
    subprocess.run(cmd, check=True, cwd=HERE)
    return out


_libs = {}


class Mutation(ctypes.Structure):
    """avo_mutation: 32-bit probability thresholds (event iff word < p32), channel masks,
    reward range, and the key / generation of the random streams."""
    _fields_ = [("seed", ctypes.c_uint64), ("generation", ctypes.c_uint64),
                ("map_flip_p32", ctypes.c_uint32), ("map_channels", ctypes.c_uint32),
                ("entry_p32", ctypes.c_uint32), ("entry_channels", ctypes.c_uint32),
                ("reward_p32", ctypes.c_uint32), ("reward_lo", ctypes.c_int32),
                ("reward_hi", ctypes.c_int32)]


def load(path: str = LIB) -> ctypes.CDLL:
    if path in _libs:
        return _libs[path]
    if not os.path.exists(path):
        if path != LIB:
            raise FileNotFoundError(path)
        build()
    lib = ctypes.CDLL(path)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.avo_create.argtypes = [I, I, I, I, I, I, I, I, I, ctypes.POINTER(P)]
    lib.avo_load_rules.argtypes = [P, I, P, P, P, P]
    lib.avo_reset.argtypes = [P, P]
    lib.avo_step.argtypes = [P, P, P, P, I, ctypes.POINTER(I)]
    lib.avo_set_rule_mode.argtypes = [P, I]
    lib.avo_set_rule_control.argtypes = [P, P, P, I, ctypes.c_uint64]
    lib.avo_site_key.argtypes = [I, ctypes.c_uint64, ctypes.c_uint64, I, I]
    lib.avo_site_key.restype = ctypes.c_uint32
    lib.avo_philox4x64.argtypes = [P, P, P]
    lib.avo_philox4x64.restype = None
    lib.avo_random_word.argtypes = [ctypes.c_uint64] * 5
    lib.avo_random_word.restype = ctypes.c_uint32
    lib.avo_mutate_maps.argtypes = [P, P, I, I, I, I, ctypes.POINTER(Mutation)]
    lib.avo_mutate_rules.argtypes = [I, I, I, I, I, P, P, P, P, P, P, P,
                                     ctypes.POINTER(Mutation)]
    lib.avo_observe.argtypes = [P, I, P]
    lib.avo_rule_features.argtypes = [P, P]
    lib.avo_get_maps.argtypes = [P, P]
    lib.avo_get_counters.argtypes = [P, P]
    lib.avo_set_counters.argtypes = [P, P]
    lib.avo_destroy.argtypes = [P]
    lib.avo_destroy.restype = None
    for f in ("avo_create", "avo_load_rules", "avo_reset", "avo_step", "avo_get_maps",
              "avo_get_counters", "avo_set_rule_mode", "avo_observe", "avo_rule_features",
              "avo_set_rule_control", "avo_mutate_maps", "avo_mutate_rules",
              "avo_set_counters"):
        getattr(lib, f).restype = I
    _libs[path] = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {code}")
        self.code = code


class Oracle:
    """One batch of environments stepped on the CPU by the oracle."""

    def __init__(self, B, H, W, C, max_rules, max_h, max_w, per_env=False, episode_len=0,
                 lib_path: str = LIB, rule_mode: int = 0):
        self.lib = load(lib_path)
        self.B, self.H, self.W, self.C = B, H, W, C
        self.max_h, self.max_w, self.per_env = max_h, max_w, bool(per_env)
        h = ctypes.c_void_p()
        rc = self.lib.avo_create(B, H, W, C, max_rules, max_h, max_w, int(bool(per_env)),
                                 episode_len, ctypes.byref(h))
        if rc != AVO_OK:
            raise OracleError("avo_create", rc)
        self.h = h
        rc = self.lib.avo_set_rule_mode(self.h, int(rule_mode))
        if rc != AVO_OK:
            raise OracleError("avo_set_rule_mode", rc)

    @classmethod
    def for_workload(cls, wl, B=None, lib_path: str = LIB, rule_mode: int = 0):
        return cls(wl.B if B is None else B, wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w,
                   wl.per_env, wl.L, lib_path=lib_path, rule_mode=rule_mode)

    def close(self):
        if getattr(self, "h", None):
            self.lib.avo_destroy(self.h)
            self.h = None

    __del__ = close

    def load_rules(self, shape, in_pat, out_pat, reward):
        shape = np.ascontiguousarray(shape, dtype=np.int32)
        in_pat = np.ascontiguousarray(in_pat, dtype=np.int8)
        out_pat = np.ascontiguousarray(out_pat, dtype=np.int8)
        reward = np.ascontiguousarray(reward, dtype=np.int32)
        R = shape.shape[1] if shape.ndim == 3 else 0
        rc = self.lib.avo_load_rules(self.h, R, _ptr(shape), _ptr(in_pat), _ptr(out_pat),
                                     _ptr(reward))
        if rc != AVO_OK:
            raise OracleError("avo_load_rules", rc)

    def set_rule_control(self, limit=None, inhibit=None, order: int = 0, seed: int = 0):
        """Rule application control: limit int32 [S][R] (0 = all), inhibit uint8 [S][R][R]
        ([q][r]: q inhibits r, q < r), order 0 row-major / 1 random, seed of the random
        index channel.  Cleared by load_rules."""
        lp = ip = None
        if limit is not None:
            limit = np.ascontiguousarray(limit, dtype=np.int32)
            lp = _ptr(limit)
        if inhibit is not None:
            inhibit = np.ascontiguousarray(inhibit, dtype=np.uint8)
            ip = _ptr(inhibit)
        rc = self.lib.avo_set_rule_control(self.h, lp, ip, int(order), int(seed))
        if rc != AVO_OK:
            raise OracleError("avo_set_rule_control", rc)

    def reset(self, init_maps):
        m = np.ascontiguousarray(init_maps, dtype=np.uint8)
        assert m.shape == (self.B, self.C, self.H, self.W), m.shape
        rc = self.lib.avo_reset(self.h, _ptr(m))
        if rc != AVO_OK:
            raise OracleError("avo_reset", rc)

    def step(self, actions, nthreads: int = 1):
        a = np.ascontiguousarray(actions, dtype=np.uint8)
        assert a.shape == (self.B,), a.shape
        rewards = np.zeros(self.B, dtype=np.float32)
        done = np.zeros(self.B, dtype=np.uint8)
        used = ctypes.c_int(0)
        rc = self.lib.avo_step(self.h, _ptr(a), _ptr(rewards), _ptr(done), nthreads,
                               ctypes.byref(used))
        if rc != AVO_OK:
            raise OracleError("avo_step", rc)
        self.threads_used = used.value
        return rewards, done

    def maps(self):
        out = np.zeros((self.B, self.C, self.H, self.W), dtype=np.uint8)
        rc = self.lib.avo_get_maps(self.h, _ptr(out))
        if rc != AVO_OK:
            raise OracleError("avo_get_maps", rc)
        return out

    def observe(self, w: int):
        out = np.zeros((self.B, self.C, w, w), dtype=np.uint8)
        rc = self.lib.avo_observe(self.h, int(w), _ptr(out))
        if rc != AVO_OK:
            raise OracleError("avo_observe", rc)
        return out

    def rule_features(self, S: int, R: int):
        out = np.zeros((S, R, 2, 2, self.C + 1, self.max_h, self.max_w), dtype=np.uint8)
        rc = self.lib.avo_rule_features(self.h, _ptr(out))
        if rc != AVO_OK:
            raise OracleError("avo_rule_features", rc)
        return out

    def set_counters(self, t):
        t = np.ascontiguousarray(t, dtype=np.int32)
        assert t.shape == (self.B,), t.shape
        rc = self.lib.avo_set_counters(self.h, _ptr(t))
        if rc != AVO_OK:
            raise OracleError("avo_set_counters", rc)

    def counters(self):
        out = np.zeros(self.B, dtype=np.int32)
        rc = self.lib.avo_get_counters(self.h, _ptr(out))
        if rc != AVO_OK:
            raise OracleError("avo_get_counters", rc)
        return out


def site_key(order: int, seed: int, n: int, b: int, pos: int, lib_path: str = LIB) -> int:
    """The oracle's index-channel value of anchor pos of env b at batch step n."""
    return int(load(lib_path).avo_site_key(order, seed, n, b, pos))


def philox4x64(ctr, key, lib_path: str = LIB):
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, np.uint64)
    load(lib_path).avo_philox4x64(_ptr(c), _ptr(k), _ptr(out))
    return out


def random_word(seed, generation, individual, stream, word, lib_path: str = LIB) -> int:
    return int(load(lib_path).avo_random_word(seed, generation, individual, stream, word))


def mutate_maps(maps, m: Mutation, lib_path: str = LIB):
    """maps uint8 [n][C][H][W] -> mutated copy (0/1)."""
    src = np.ascontiguousarray(maps, dtype=np.uint8)
    dst = np.empty_like(src)
    n, C, H, W = src.shape
    rc = load(lib_path).avo_mutate_maps(_ptr(src), _ptr(dst), n, C, H, W, ctypes.byref(m))
    if rc != AVO_OK:
        raise OracleError("avo_mutate_maps", rc)
    return dst


def mutate_rules(shape, in_pat, out_pat, reward, m: Mutation, lib_path: str = LIB):
    """Rules in the av_load_rules layout -> mutated (in_pat, out_pat, reward)."""
    shape = np.ascontiguousarray(shape, dtype=np.int32)
    ip = np.ascontiguousarray(in_pat, dtype=np.int8)
    op = np.ascontiguousarray(out_pat, dtype=np.int8)
    rw = np.ascontiguousarray(reward, dtype=np.int32)
    S, R, C1, mh, mw = ip.shape
    ip2, op2, rw2 = np.empty_like(ip), np.empty_like(op), np.empty_like(rw)
    rc = load(lib_path).avo_mutate_rules(S, R, C1 - 1, mh, mw, _ptr(shape), _ptr(ip), _ptr(op),
                                         _ptr(rw), _ptr(ip2), _ptr(op2), _ptr(rw2),
                                         ctypes.byref(m))
    if rc != AVO_OK:
        raise OracleError("avo_mutate_rules", rc)
    return ip2, op2, rw2


def run(wl, maps, rules, actions, nthreads: int = 1, B=None, lib_path: str = LIB,
        rule_mode: int = 0, control=None):
    """Step a workload's arrays for len(actions) steps; returns the per-step trajectory
    (maps [T][B][C][H][W], rewards [T][B], done [T][B]).  control: None or
    (limit, inhibit, order, seed) for set_rule_control."""
    B = maps.shape[0] if B is None else B
    o = Oracle.for_workload(wl, B=B, lib_path=lib_path, rule_mode=rule_mode)
    o.load_rules(*rules)
    if control is not None:
        o.set_rule_control(*control)
    o.reset(maps)
    T = actions.shape[0]
    out_maps = np.zeros((T,) + maps.shape, dtype=np.uint8)
    out_r = np.zeros((T, B), dtype=np.float32)
    out_d = np.zeros((T, B), dtype=np.uint8)
    for t in range(T):
        out_r[t], out_d[t] = o.step(actions[t], nthreads)
        out_maps[t] = o.maps()
    o.close()
    return out_maps, out_r, out_d
