"""The selector's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

`tests/sanitize/selector_driver.cpp` is built with g++ together with the
selector's source, with both sanitizers and no recovery, and fed random and
extreme workloads and parameters (dimensions near INT32_MAX, rho and the
split cost near INT64_MAX, c_max up to INT32_MAX, invalid fields).  The run
must end cleanly, and every entry point must return what the shared
library returns for the same case: the same candidate, table, split count
and candidate internals, or the same error.
"""
import ctypes
import os
import random
import shutil
import subprocess

import numpy as np
import pytest

from paper_2609_07536_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
I32 = 2**31 - 1
I64 = 2**63 - 1

PARAM_FIELDS = ["tile_m", "tile_n", "comm_tile_m", "comm_tile_n", "occ_comp", "occ_comm",
                "num_cus", "c_min", "c_max", "groups", "rho_ref_num", "rho_ref_den", "k_ref",
                "tile_m_ref", "tile_n_ref", "d_ref", "split_axis", "drain", "rho_kh", "topk_ref",
                "comm_tile_n_ref", "readiness", "comm_tile_m_last", "split_cost_num",
                "split_cost_den"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("sanitize") / "selector_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2609_07536_amd", "csrc", "selector.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "selector_driver.cpp"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return out


def _params(**kw):
    p = dict(tile_m=256, tile_n=256, comm_tile_m=64, comm_tile_n=1024, occ_comp=1, occ_comm=1,
             num_cus=256, c_min=0, c_max=64, groups=1, rho_ref_num=159, rho_ref_den=100,
             k_ref=704, tile_m_ref=256, tile_n_ref=256, d_ref=1, split_axis=0, drain=0,
             rho_kh=0, topk_ref=6, comm_tile_n_ref=1024, readiness=0, comm_tile_m_last=0,
             split_cost_num=0, split_cost_den=1)
    p.update(kw)
    return p


def _random_case(rnd):
    E = rnd.randint(1, 64)
    topk = rnd.randint(1, min(E, 8))
    T = rnd.randint(0, 40000)
    L = rnd.randint(1, 4)
    H = 8 * L * rnd.randint(1, 512)
    I = 8 * rnd.randint(1, 200)
    counts = None
    if rnd.random() < 0.8:
        w = np.array([rnd.random() ** 3 for _ in range(E)])
        c = np.floor(w / w.sum() * T * topk).astype(np.int64)
        c[0] += T * topk - c.sum()
        counts = [int(v) for v in c]
    p = _params(tile_m=rnd.choice([64, 128, 256]), tile_n=rnd.choice([64, 128, 256]),
                comm_tile_m=rnd.choice([16, 64, 128]), occ_comp=rnd.randint(1, 3),
                occ_comm=rnd.randint(1, 3), num_cus=rnd.choice([8, 108, 256]),
                c_min=rnd.choice([0, 1]), c_max=rnd.randint(1, 80),
                rho_ref_num=rnd.randint(1, 100000), rho_ref_den=rnd.randint(1, 10000),
                split_axis=rnd.choice([0, 0, 1]), drain=rnd.choice([0, 1, 2]),
                rho_kh=rnd.choice([0, 1]), d_ref=rnd.choice([1, 4]))
    if p["split_axis"] == 0 and p["drain"] != 2 and rnd.random() < 0.3:
        p["readiness"] = 1
    if p["readiness"] == 0 and p["drain"] != 2 and p["split_axis"] == 0 and rnd.random() < 0.3:
        p["comm_tile_m_last"] = p["comm_tile_m"] // 2
    if p["readiness"] == 0 and rnd.random() < 0.4:
        p["split_cost_num"], p["split_cost_den"] = rnd.choice([(43, 100), (1, 3), (7919, 257)])
    wl = dict(T=T, H=H, I=I, E=E, topk=topk, splits=L, ranks=rnd.choice([1, 2]), rows=0,
              counts=counts)
    return wl, p, rnd.randint(0, p["c_max"]), 1, rnd.randint(1, 4)


def _extreme_cases():
    """Dimensions, rates and ranges at the ends of their types, and invalid
    fields: each must come back as a result or an error, never as undefined
    behaviour or a hang."""
    base = dict(T=16384, H=2048, I=704, E=32, topk=6, splits=2, ranks=1, rows=0,
                counts=[3072] * 32)
    cases = []
    big_counts = dict(base, E=1024, counts=[I32] * 1024, T=I32, topk=1)
    for wl, p in [
        (base, _params(c_max=I32)),                                   # huge candidate range
        (base, _params(c_min=1, c_max=I32, readiness=1)),
        (base, _params(c_max=I32, drain=2, split_axis=1, split_cost_num=43, split_cost_den=100)),
        (big_counts, _params(tile_m=1, tile_n=1)),                    # W_comp near 2^41
        (big_counts, _params(tile_m=1, tile_n=1, readiness=1, c_min=1)),  # V beyond 2^20
        (big_counts, _params(tile_m=1, tile_n=1, drain=2)),
        (dict(base, H=I32, I=1), _params(tile_n=1, comm_tile_n=1)),
        (dict(base, I=I32), _params()),
        (base, _params(rho_ref_num=I64, rho_ref_den=1)),               # rho near 2^63
        (base, _params(rho_ref_num=1, rho_ref_den=I64)),
        (base, _params(rho_ref_num=I64, rho_ref_den=I64 - 1, rho_kh=1)),
        (base, _params(split_cost_num=I64, split_cost_den=1)),
        (base, _params(split_cost_num=1, split_cost_den=I64)),
        (base, _params(split_cost_num=I64, split_cost_den=I64 - 2, drain=2)),
        (base, _params(occ_comp=I32, occ_comm=I32, num_cus=I32)),     # o G beyond int32
        (base, _params(occ_comp=65536, num_cus=32768)),
        (base, _params(num_cus=1, c_min=1)),                          # no legal candidate
        (dict(base, splits=I32), _params()),                          # too many splits
        (dict(base, splits=1 << 20), _params(c_max=2)),
        (dict(base, T=0, counts=[0] * 32), _params(drain=2)),         # empty batch
        (dict(base, counts=None), _params(comm_tile_m_last=I32)),
        (base, _params(comm_tile_m=I32, comm_tile_n=I32)),
        (base, _params(k_ref=I32, tile_m_ref=I32, tile_n_ref=I32, d_ref=1)),
        (dict(base, ranks=I32), _params(d_ref=1)),
        (base, _params(c_min=-1)),                                    # invalid fields
        (base, _params(c_max=-5)),
        (base, _params(drain=-1)),
        (base, _params(split_cost_num=-3)),
        (base, _params(split_cost_num=2, split_cost_den=0)),
        (base, _params(split_cost_num=2, split_cost_den=5, readiness=1)),
        (dict(base, counts=[-1] + [3072] * 31), _params()),
        (dict(base, T=-1), _params()),
    ]:
        cases.append((wl, p, 5, 1, 4))
        cases.append((wl, p, 0, 1, 2))
    cases.append((base, _params(), 0, 1, 1024))                       # the widest L range
    cases.append((base, _params(drain=2, split_axis=1, split_cost_num=43, split_cost_den=100),
                  0, 1, 1024))
    cases.append((base, _params(), 3, 1, 1025))                       # L range too wide
    cases.append((base, _params(), 3, 0, 2))
    return cases


def _line(wl, p, C, l_min, l_max):
    counts = wl["counts"]
    head = [wl["T"], wl["H"], wl["I"], wl["E"], wl["topk"], wl["splits"], wl["ranks"],
            wl["rows"], 1 if counts is not None else 0] + (list(counts) if counts else [])
    return " ".join(str(v) for v in head + [p[f] for f in PARAM_FIELDS] + [C, l_min, l_max])


def _library_line(wl, p, C, l_min, l_max):
    """The driver's output for one case, from the shared library."""
    L = B.lib()
    w, keep = B.make_workload(wl["T"], wl["H"], wl["I"], wl["E"], wl["topk"], wl["splits"],
                              wl["counts"], rows=wl["rows"], ranks=wl["ranks"])
    sp = B.SelectParams(**p)
    part = B.Partition()
    r = L.moe_select_partition(ctypes.byref(w), ctypes.byref(sp), ctypes.byref(part))
    s = f"part {r}"
    if r >= 0:
        s += (f" {part.C} {part.R} {part.P} {part.delta_comp} {part.T_num} {part.T_den}"
              f" {part.W_comp} {part.W_comm}")
    span = p["c_max"] - p["c_min"]
    n = span + 1 if 0 <= span < 100000 else 0
    buf = (ctypes.c_int64 * max(n, 1))()
    den = ctypes.c_int64(0)
    re = L.moe_select_evaluate(ctypes.byref(w), ctypes.byref(sp), buf, n, ctypes.byref(den))
    s += f" | eval {re}"
    if re > 0:
        s += f" {den.value}" + "".join(f" {buf[i]}" for i in range(re))
    sp2 = B.Partition()
    Lout = ctypes.c_int32(0)
    rs = L.moe_select_partition_splits(ctypes.byref(w), ctypes.byref(sp), l_min, l_max,
                                       ctypes.byref(sp2), ctypes.byref(Lout))
    s += f" | splits {rs}"
    if rs >= 0:
        s += f" {Lout.value} {sp2.T_num} {sp2.T_den}"
    cn, cd = ctypes.c_int64(0), ctypes.c_int64(0)
    k = L.moe_select_candidate(ctypes.byref(w), ctypes.byref(sp), C, ctypes.byref(cn),
                               ctypes.byref(cd), None, None, 0)
    s += f" | cand {k}"
    if k > 0:
        A, F = (ctypes.c_int64 * k)(), (ctypes.c_int64 * k)()
        k2 = L.moe_select_candidate(ctypes.byref(w), ctypes.byref(sp), C, ctypes.byref(cn),
                                    ctypes.byref(cd), A, F, k)
        s += f" {k2} {cn.value} {cd.value}" + "".join(f" {A[i]} {F[i]}" for i in range(k2))
    return s


def test_selector_under_sanitizers(driver):
    rnd = random.Random(5)
    cases = [_random_case(rnd) for _ in range(400)] + _extreme_cases()
    stdin = "\n".join(_line(*c) for c in cases) + "\n"
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([driver], input=stdin, capture_output=True, text=True, timeout=600,
                       env=env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, \
        r.stderr[-4000:]
    got = r.stdout.splitlines()
    assert len(got) == len(cases)
    n_ok = 0
    for c, line in zip(cases, got):
        assert line == _library_line(*c), _line(*c)
        n_ok += not line.startswith("part -")
    assert n_ok > 300
    # the extreme cases end as results or errors, and the huge candidate
    # ranges as results: the selection stops at the first illegal C
    ext = got[-(len(_extreme_cases())):]
    assert ext[0].startswith("part 0 ") and " | eval -1" in ext[0]
    assert all(" | splits -1" in line for line in ext[-2:])
