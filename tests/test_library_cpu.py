"""Host-side checks of libmts (no GPU): the library loads, exports every
symbol include/mts.h declares, sizes every workload and rejects
configurations outside its documented limits."""
import copy
import math
import os
import re

import pytest

from paper_2608_16336_amd import mts
from workloads import PRESETS, preset

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "mts.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mts_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = mts.load_library()
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(mts.EXPORTED)


def test_binding_fails_loudly_without_library(tmp_path):
    saved = mts._lib
    mts._lib = None
    try:
        with pytest.raises(OSError):
            mts.load_library(str(tmp_path / "missing.so"))
    finally:
        mts._lib = saved


@pytest.mark.parametrize("name", sorted(PRESETS))
def test_state_bytes(name):
    c = preset(name)
    R = sum(g["n_replicas"] for g in c["groups"])
    n_slots = R * c["n_instances"] * c["slots_per_instance"]
    b = mts.mts_state_bytes(c)
    # slot arrays (13 B per slot), at most 2 GiB of pre-sampled arrivals, a
    # finish wheel of at most 512 buckets per replica and small tables
    a = c["arrival"]
    cv = a.get("cv", 0.0) if a["kind"] == "gamma_poisson" else 0.0
    wcap = min(2048, math.ceil((2 * a["mean"] * (1 + cv) + 24) / 16) * 16)
    wheel = R * 512 * wcap * 4 + 2**20
    assert 13 * n_slots <= b < 13 * n_slots + wheel + 2136 * 2**20


def _bad(**over):
    c = preset("tiny")
    for k, v in over.items():
        if k.startswith("g_"):
            c["groups"][0][k[2:]] = v
        else:
            c[k] = v
    return c


@pytest.mark.parametrize("cfg", [
    _bad(g_K=0), _bad(g_K=11), _bad(n_instances=0), _bad(n_instances=257),
    _bad(slots_per_instance=96), _bad(slots_per_instance=8192), _bad(slots_per_instance=0),
    _bad(block_tokens=12), _bad(block_tokens=0), _bad(kv_blocks=0), _bad(kv_blocks=(1 << 21) + 1),
    _bad(theta_den=0), _bad(theta_num=-1), _bad(mig_interval=0), _bad(mig_stage_blocks=0),
    _bad(mig_max_pairs=3), _bad(headroom_decay=1.5), _bad(headroom_base=-1.0),
    _bad(prompt=dict(kind="uniform_int", lo=0, hi=10)),
    _bad(prompt=dict(kind="uniform_int", lo=60000, hi=65000)),  # prompt + output > 65535 tokens
    _bad(output=dict(kind="geometric", mean=0.5)),
    _bad(arrival=dict(kind="poisson", mean=0.0)),
    _bad(g_n_replicas=0),
    # Section 6.5 extensions: the same limits the oracle enforces
    _bad(adaptive=dict(epoch=10, step_up=1, step_down=1, max=256 * 600, margin=257, slo=[5])),
    _bad(adaptive=dict(epoch=10, step_up=1, step_down=1, max=(1 << 29) // 10 + 1, margin=0, slo=[5])),
    _bad(adaptive=dict(epoch=(1 << 16) + 1, step_up=1, step_down=1, max=256 * 600, margin=0, slo=[5])),
    _bad(adaptive=dict(epoch=10, step_up=1, step_down=1, max=256 * 600, margin=0, slo=[0])),
    _bad(adaptive=dict(epoch=10, step_up=1, step_down=1, max=256 * 600, margin=0, slo=[1 << 21])),
    _bad(adaptive=dict(epoch=10, step_up=1, step_down=1, max=100, margin=0, slo=[5])),  # below Eq. 3's H_0
], ids=lambda c: "bad")
def test_invalid_configs_are_rejected(cfg):
    with pytest.raises(mts.MtsError) as e:
        mts.mts_state_bytes(cfg)
    assert e.value.code == -1


def test_abi_version_is_checked():
    c, g = mts.make_cfg(preset("tiny"))
    c.abi_version = 99
    import ctypes
    n = ctypes.c_size_t(0)
    assert mts.load_library().mts_state_bytes(ctypes.byref(c), ctypes.byref(n)) == -1


def test_strerror():
    L = mts.load_library()
    assert L.mts_strerror(0) == b"ok"
    assert b"invalid" in L.mts_strerror(-1)


def test_adaptive_limits_accept_what_the_oracle_accepts():
    import oracle
    c = _bad(adaptive=dict(epoch=1 << 16, step_up=2**32 - 1, step_down=2**32 - 1, max=(1 << 29) // 10,
                           margin=256, slo=[1, 1 << 20]), promotion=dict(period=2**32 - 1, age=[2**32 - 1] * 10))
    assert mts.mts_state_bytes(c) > 0
    oracle.Oracle(c).close()
