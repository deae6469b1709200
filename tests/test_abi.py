"""The C ABI boundary without a GPU: the library loads, exports every function that
include/autoverse.h declares, and rejects bad arguments on the host before any device
work, with a message."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2407_04221_amd as av

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
           if f.endswith(".h")]


def declared_functions():
    names = set()
    for h in HEADERS:
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(av_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(av.LIB_PATH):
        from paper_2407_04221_amd import build
        build.build()
    return av.load_library()


def test_every_declared_function_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 15
    assert set(names) == set(av.ABI_SYMBOLS)
    out = subprocess.run(["nm", "-D", "--defined-only", av.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (av_[a-z_0-9]+)$", out, flags=re.M))
    missing = set(names) - exported
    assert not missing, f"not exported: {missing}"
    for n in names:
        assert hasattr(lib, n)


def test_no_torch_types_in_the_abi():
    for h in HEADERS:
        text = open(h).read()
        assert "torch" not in text.lower().replace("torch tensors", "")
        assert "#include <hip" not in text      # plain C types only


def _cfg(**kw):
    base = dict(num_envs=4, height=16, width=16, channels=6, max_rules=8, max_pat_h=3,
                max_pat_w=3, per_env_rules=0, max_episode_steps=0, device=0, engine=0,
                rule_mode=0, stream=None)
    base.update(kw)
    return av.av_config(*[base[f] for f, _ in av.av_config._fields_])


@pytest.mark.parametrize("bad", [
    dict(num_envs=0), dict(height=0), dict(width=65), dict(height=65), dict(channels=3),
    dict(channels=32), dict(max_rules=-1), dict(max_rules=253), dict(max_pat_h=0),
    dict(max_pat_w=17), dict(per_env_rules=2), dict(max_episode_steps=-1), dict(engine=9),
    dict(engine=6), dict(engine=-1),
    # the group engine: parallel rule order, maps of at most 32 x 32, (R + 4) x pattern cells
    # <= 254
    dict(engine=5, rule_mode=1), dict(engine=5, height=33, width=20),
    dict(engine=5, max_rules=25), dict(engine=5, max_pat_h=16, max_pat_w=16, max_rules=1),
    # the rows engine takes at most 60 loaded rules and its LDS set within 64 KiB
    dict(engine=4, max_rules=61), dict(engine=4, height=64, width=64, channels=31, max_rules=60),
    # lane16 needs maps of at most 16 x 16 and one shared rule set
    dict(engine=2, height=32, width=32), dict(engine=2, per_env_rules=1),
    dict(rule_mode=2), dict(rule_mode=-1),
    # the wave engine's LDS working set over 64 KiB (the generic engine's fits)
    dict(engine=3, channels=31, max_rules=140),
    # one environment's LDS working set over 64 KiB
    dict(height=64, width=64, channels=31, max_rules=252),
])
def test_create_rejects_bad_config(lib, bad):
    cfg = _cfg(**bad)
    h = ctypes.c_void_p(1234)
    rc = lib.av_create_batch(ctypes.byref(cfg), ctypes.byref(h))
    assert rc == av.AV_EINVAL
    assert h.value is None
    assert av.av_last_error()


def test_null_arguments_are_rejected(lib):
    h = ctypes.c_void_p()
    assert lib.av_create_batch(None, ctypes.byref(h)) == av.AV_EINVAL
    cfg = _cfg()
    assert lib.av_create_batch(ctypes.byref(cfg), None) == av.AV_EINVAL
    assert lib.av_step(None, None, None, None) == av.AV_EINVAL
    assert "NULL" in av.av_last_error()
    assert lib.av_step_n(None, 1, None, None, None) == av.AV_EINVAL
    assert lib.av_load_rules(None, 0, None, None, None, None) == av.AV_EINVAL
    assert lib.av_reset(None, None) == av.AV_EINVAL
    assert lib.av_get_maps(None, None) == av.AV_EINVAL
    assert lib.av_observe(None, 5, None) == av.AV_EINVAL
    assert lib.av_rule_features(None, None) == av.AV_EINVAL
    assert lib.av_set_rule_control(None, None, None, 0, 0) == av.AV_EINVAL
    assert lib.av_step_observe(None, 1, None, None, None, 5, None) == av.AV_EINVAL
    m = av.mutation()
    assert lib.av_mutate_maps(None, None, 1, 4, 4, 4, m, 0, None) == av.AV_EINVAL
    assert lib.av_mutate_maps(None, None, 1, 4, 4, 4, None, 0, None) == av.AV_EINVAL
    assert lib.av_mutate_maps(None, None, -1, 4, 4, 4, m, 0, None) == av.AV_EINVAL
    assert lib.av_mutate_maps(None, None, 1, 32, 4, 4, m, 0, None) == av.AV_EINVAL
    assert lib.av_mutate_rules(1, 1, 4, 3, 3, None, None, None, None, None, None, None, m, 0,
                               None) == av.AV_EINVAL
    assert lib.av_mutate_rules(1, 1, 4, 17, 3, None, None, None, None, None, None, None, m, 0,
                               None) == av.AV_EINVAL
    assert lib.av_search_create(None, None) == av.AV_EINVAL
    assert lib.av_search_load_rules(None, 0, None, None, None, None) == av.AV_EINVAL
    assert lib.av_search_begin(None, None) == av.AV_EINVAL
    assert lib.av_search_expand(None, 1, None) == av.AV_EINVAL
    assert lib.av_search_frontier(None, None, None, None) == av.AV_EINVAL
    assert lib.av_search_destroy(None) == av.AV_OK
    bad = av.mutation(reward_lo=2, reward_hi=1)
    assert lib.av_mutate_rules(0, 0, 4, 3, 3, None, None, None, None, None, None, None, bad, 0,
                               None) == av.AV_EINVAL
    assert lib.av_state_ptr(None) is None
    info = av.av_info()
    assert lib.av_get_info(None, ctypes.byref(info)) == av.AV_EINVAL
    n = ctypes.c_size_t(0)
    assert lib.av_get_state(None, None, ctypes.byref(n)) == av.AV_EINVAL
    assert lib.av_set_state(None, None, 0) == av.AV_EINVAL
    assert lib.av_set_stream(None, None) == av.AV_EINVAL
    assert lib.av_destroy_batch(None) == av.AV_OK


def test_last_error_is_cleared_by_a_successful_call(lib):
    lib.av_step(None, None, None, None)
    assert av.av_last_error()
    assert lib.av_destroy_batch(None) == av.AV_OK
    assert av.av_last_error() == ""


def test_missing_library_fails_loudly():
    """No fallback: without libautoverse.so the binding raises instead of computing anything."""
    import subprocess
    import sys
    code = ("import paper_2407_04221_amd as av\n"
            "try:\n    av.load_library('/nonexistent/libautoverse.so')\n"
            "except RuntimeError as e:\n    print('raised', e)\n")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    assert out.stdout.startswith("raised"), out.stdout + out.stderr


def test_product_and_oracle_share_no_code():
    """The library's sources and binding never name the oracle, the oracle never names the
    library's sources, and the built library needs no oracle symbol."""
    import re
    import subprocess
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    pkg = os.path.join(root, "paper_2407_04221_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h", ".inc")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"\bimport oracle\b|from oracle\b|avo_|avo\.h", text), f
    for f in os.listdir(os.path.join(root, "oracle")):
        if f.endswith((".c", ".h", ".py")):
            text = open(os.path.join(root, "oracle", f)).read()
            assert "csrc" not in text and "paper_2407_04221_amd" not in text.replace(
                "from paper_2407_04221_amd import inputs", ""), f
    lib = av.LIB_PATH
    if os.path.exists(lib):
        und = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True,
                             text=True).stdout
        assert "avo_" not in und
