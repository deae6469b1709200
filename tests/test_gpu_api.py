"""The C ABI on a GPU: state errors, rule validation, checkpoint/resume, determinism,
the packed state layout, and the exhaustive 4x4 batches run through the HIP path."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2407_04221_amd as av
from gpu_util import gpu_run, require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu


def small():
    return inputs.Workload("api", 11, B=19, H=9, W=13, C=5, R=4, shapes=((3, 3), (1, 2)),
                           p_dc=0.5, per_env=False, T=12, L=5)


def test_step_before_rules_and_reset_is_a_state_error():
    require_gpu()
    import torch
    wl = small()
    b = av.Batch.for_workload(wl)
    acts = torch.zeros(wl.B, dtype=torch.uint8, device="cuda")
    with pytest.raises(av.AvError) as e:
        b.step(acts)
    assert e.value.status == av.AV_ESTATE
    maps, rules, _ = inputs.make_all(wl, 0)
    b.load_rules(*rules)
    with pytest.raises(av.AvError) as e:
        b.step(acts)
    assert e.value.status == av.AV_ESTATE
    b.reset(maps)
    b.step(acts)
    lib = av.load_library()          # k = 0 straight through the C ABI
    rc = lib.av_step_n(b.h, 0, ctypes.c_void_p(acts.data_ptr()),
                       ctypes.c_void_p(b.rewards.data_ptr()), ctypes.c_void_p(b.done.data_ptr()))
    assert rc == av.AV_EINVAL and "k must be" in av.av_last_error()
    b.close()


def test_rule_validation():
    require_gpu()
    wl = small()
    b = av.Batch.for_workload(wl)
    shape, ip, op, rw = inputs.make_rules(wl, 0)
    bad = ip.copy()
    bad[0, 1, 2, 0, 0] = 2
    with pytest.raises(av.AvError) as e:
        b.load_rules(shape, bad, op, rw)
    assert e.value.status == av.AV_EINVAL and "pattern value" in e.value.message
    big = shape.copy()
    big[0, 0] = (4, 1)            # larger than max_pat_h = 3
    with pytest.raises(av.AvError):
        b.load_rules(big, ip, op, rw)
    huge = rw.copy()
    huge[0, 0] = 1 << 20          # |reward| x anchors over 2^24
    with pytest.raises(av.AvError) as e:
        b.load_rules(shape, ip, op, huge)
    assert "2^24" in e.value.message
    too_many = (np.zeros((1, wl.R + 1, 2), np.int32) + 1,
                np.full((1, wl.R + 1, wl.C + 1, 3, 3), -1, np.int8),
                np.full((1, wl.R + 1, wl.C + 1, 3, 3), -1, np.int8),
                np.zeros((1, wl.R + 1), np.int32))
    with pytest.raises(av.AvError):
        b.load_rules(*too_many)
    b.load_rules(shape, ip, op, rw)
    b.close()


@pytest.mark.parametrize("engine", ["generic", "wave", "rows", "auto"])
def test_checkpoint_resume_is_bit_identical(engine):
    require_gpu()
    import torch
    wl = inputs.WORKLOADS["c4"].with_(B=300, T=40, L=9)
    maps, rules, actions = inputs.make_all(wl, 5, "dense")
    acts = torch.from_numpy(actions).cuda()
    b = av.Batch.for_workload(wl, engine=engine)
    b.load_rules(*rules)
    b.reset(maps)
    b.step_n(acts[:17])
    blob = b.get_state()
    r1, d1 = b.step_n(acts[17:])
    m1 = b.maps().cpu().numpy()
    c = av.Batch.for_workload(wl, engine=engine)
    c.load_rules(*rules)
    c.set_state(blob)
    r2, d2 = c.step_n(acts[17:])
    assert torch.equal(r1, r2) and torch.equal(d1, d2)
    assert np.array_equal(m1, c.maps().cpu().numpy())
    other = av.Batch(wl.B + 1, wl.H, wl.W, wl.C, wl.R, 3, 3)
    with pytest.raises(av.AvError):
        other.set_state(blob)
    for x in (b, c, other):
        x.close()


@pytest.mark.parametrize("engine", ["generic", "wave", "rows", "auto"])
def test_two_runs_are_identical(engine):
    require_gpu()
    wl = inputs.WORKLOADS["c2"].with_(B=150, T=30)
    maps, rules, actions = inputs.make_all(wl, 4, "dense")
    a = gpu_run(wl, maps, rules, actions, engine=engine, mode="step_n", chunk=30)
    b = gpu_run(wl, maps, rules, actions, engine=engine, mode="step_n", chunk=30)
    for x, y in zip(a[1:4], b[1:4]):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("W", [5, 16, 17, 32, 33, 64])
def test_packed_state_layout(W):
    require_gpu()
    import torch
    wl = inputs.Workload("lay", 12, B=6, H=7, W=W, C=4, R=1, shapes=((1, 1),), p_dc=0.5,
                         per_env=False, T=1)
    maps, rules, _ = inputs.make_all(wl, 0)
    b = av.Batch.for_workload(wl)
    b.load_rules(*rules)
    b.reset(maps)
    info = b.info
    rb = info["row_bytes"]
    assert rb == (2 if W <= 16 else 4 if W <= 32 else 8)
    n = info["state_bytes"]
    raw = torch.empty(n, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    hip.hipMemcpy.restype = ctypes.c_int
    HIP_MEMCPY_DEVICE_TO_DEVICE = 3
    assert hip.hipMemcpy(raw.data_ptr(), b.state_ptr(), n, HIP_MEMCPY_DEVICE_TO_DEVICE) == 0
    torch.cuda.synchronize()
    host = raw.cpu().numpy()
    words = host.view({2: np.uint16, 4: np.uint32, 8: np.uint64}[rb]).reshape(wl.C, wl.B, wl.H)
    bits = (words[..., None].astype(np.uint64) >> np.arange(W, dtype=np.uint64)) & 1
    np.testing.assert_array_equal(bits.transpose(1, 0, 2, 3).astype(np.uint8), maps)
    np.testing.assert_array_equal(b.maps().cpu().numpy(), maps)
    b.close()


@pytest.mark.parametrize("engine", ["generic", "wave", "rows", "auto"])
def test_exhaustive_4x4_rules_against_oracle(engine):
    """Every 4x4 goal plane x a sample of tri-valued 1x2 / 2x1 rules, 65536 envs each."""
    require_gpu()
    k = np.arange(1 << 16, dtype=np.int64)
    planes = ((k[:, None] >> np.arange(16)[None, :]) & 1).reshape(-1, 4, 4).astype(np.uint8)
    B = planes.shape[0]
    maps = np.zeros((B, 4, 4, 4), np.uint8)
    maps[:, 3] = planes
    maps[:, 2, 3, 3] = 1
    wl = inputs.Workload("b3", 13, B=B, H=4, W=4, C=4, R=1, shapes=((1, 2), (2, 1)),
                         p_dc=0.0, per_env=False, T=1)     # pattern arrays 2 x 2
    g = np.random.default_rng(3)
    for n, m in ((1, 2), (2, 1)):
        for _ in range(8):
            ip = np.full((1, 1, 5, 2, 2), -1, np.int8)
            op = np.full((1, 1, 5, 2, 2), -1, np.int8)
            ip[0, 0, 3, :n, :m] = g.integers(-1, 2, size=(n, m))
            op[0, 0, 3, :n, :m] = g.integers(-1, 2, size=(n, m))
            rules = (np.array([[[n, m]]], np.int32), ip, op, np.array([[1]], np.int32))
            acts = np.zeros((1, B), np.uint8)
            say(f"[b3] {n}x{m} engine={engine}")
            want = oracle.run(wl, maps, rules, acts, nthreads=8)
            _, final, r, d, _ = gpu_run(wl, maps, rules, acts, engine=engine, mode="step")
            np.testing.assert_array_equal(final, want[0][0])
            np.testing.assert_array_equal(r, want[1])
            np.testing.assert_array_equal(d, want[2])


@pytest.mark.parametrize("engine", ["generic", "wave", "rows", "auto"])
def test_exhaustive_4x4_moves_against_oracle(engine):
    """Every 4x4 wall plane x 3 player cells x 5 actions, no loaded rules."""
    require_gpu()
    k = np.arange(1 << 16, dtype=np.int64)
    walls = ((k[:, None] >> np.arange(16)[None, :]) & 1).reshape(-1, 4, 4).astype(np.uint8)
    B = walls.shape[0]
    wl = inputs.Workload("b3m", 14, B=B, H=4, W=4, C=4, R=0, shapes=((1, 1),), p_dc=0.0,
                         per_env=False, T=1)
    empty = (np.zeros((1, 0, 2), np.int32), np.zeros((1, 0, 5, 1, 1), np.int8),
             np.zeros((1, 0, 5, 1, 1), np.int8), np.zeros((1, 0), np.int32))
    for py, px in ((0, 0), (1, 2), (3, 1)):
        maps = np.zeros((B, 4, 4, 4), np.uint8)
        maps[:, 1] = walls
        maps[:, 2, py, px] = 1
        for a in range(6):
            acts = np.full((1, B), a, np.uint8)
            want = oracle.run(wl, maps, empty, acts, nthreads=8)
            _, final, r, d, _ = gpu_run(wl, maps, empty, acts, engine=engine, mode="step")
            np.testing.assert_array_equal(final, want[0][0], err_msg=f"({py},{px}) a={a}")
