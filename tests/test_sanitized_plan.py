"""The plan builder and allocator under the address and undefined-behaviour
sanitizers: tests/native/plan_driver.cpp and pfx_plan.cpp built with g++
(no HIP), run over valid batches (the five workloads' shapes, small mixed
cases, G from 1 to 16, short pieces) and malformed ones (every error the
ABI tests reach).  The driver must exit cleanly, report what the library
reports through ctypes, and the sanitizers must find nothing."""

from __future__ import annotations

import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2608_25523_amd import binding as B
from paper_2608_25523_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def case_text(b, mode=B.PFX_MODE_MIXED, piece_steps=0, workers=0, hq=None, num_pages=None, d=None,
              agent=None, slen=None, q_indptr=None, pids=None):
    pind, pids0, plen = b.prefix_csr()
    sind, sids = b.suffix_csr()
    pids = pids0 if pids is None else np.asarray(pids, np.int32)
    agent = b.agent if agent is None else np.asarray(agent, np.int32)
    slen = b.suffix_len if slen is None else np.asarray(slen, np.int32)
    q_indptr = b.q_indptr() if q_indptr is None else np.asarray(q_indptr, np.int32)
    hdr = [num_pages or b.num_pages, b.num_kv_heads, d or b.head_dim, hq or b.num_q_heads, mode, piece_steps, workers]
    rows = [hdr, [len(plen)], plen, pind, pids, [len(agent)], agent, sind, sids, slen, q_indptr]
    return "\n".join(" ".join(str(int(x)) for x in r) for r in rows) + "\n"


def cases():
    out = []
    for cfg in (1, 2, 3, 4):
        b = W.config_batch(cfg)
        out.append((b, {}))
    small = W.make_batch(11, num_q_heads=8, num_kv_heads=2, head_dim=64, num_pages=64, prefix_len=[40, 17],
                         agent=[0, 1, 0, -1, 1], suffix_len=[5, 20, 33, 3, 16], n_rows=[1, 1, 33, 3, 2])
    out += [(small, {}), (small, dict(piece_steps=1, workers=3)), (small, dict(hq=2)), (small, dict(hq=32)),
            (small, dict(mode=B.PFX_MODE_DECODE)),                   # n_r > 1 in decode mode: EINVAL
            (small, dict(num_pages=20)),                             # Eq. (2): ENOMEM
            (small, dict(d=96)), (small, dict(hq=6)),                # EUNSUPPORTED
            (small, dict(agent=[0, 1, 0, 5, 1])),                    # ERANGE
            (small, dict(slen=[5, 20, 33, 3, 40])),                  # page count mismatch: EINVAL
            (small, dict(q_indptr=[0, 1, 2, 35, 39, 41])),           # n_r > L_r: ERANGE
            (small, dict(pids=np.r_[small.prefix_csr()[1][:-1], small.prefix_csr()[1][0]]))]  # page twice
    return out


def library_result(b, kw):
    pool = B.make_pool(kw.get("num_pages") or b.num_pages, b.num_kv_heads, kw.get("d") or b.head_dim)
    pind, pids, plen = b.prefix_csr()
    if kw.get("pids") is not None:
        pids = np.asarray(kw["pids"], np.int32)
    sind, sids = b.suffix_csr()
    agent = kw.get("agent", b.agent)
    slen = kw.get("slen", b.suffix_len)
    qind = kw.get("q_indptr", b.q_indptr())
    try:
        p = B.pfx_plan_create(pool, pind, pids, plen, agent, sind, sids, slen, qind, kw.get("hq") or b.num_q_heads,
                              kw.get("mode", B.PFX_MODE_MIXED), decode_workers=kw.get("workers", 0),
                              piece_steps=kw.get("piece_steps", 0))
    except B.PfxError as e:
        return e.code, None
    s = p.stats()
    return 0, (s.num_tokens, s.num_items, s.num_decode_pieces, s.num_partial_rows, s.pages_needed,
               s.workspace_bytes)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is not installed")
def test_plan_builder_under_sanitizers(tmp_path):
    exe = tmp_path / "plan_driver"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "native", "plan_driver.cpp"),
           os.path.join(ROOT, "paper_2608_25523_amd", "csrc", "pfx_plan.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    cs = cases()
    inp = tmp_path / "cases.txt"
    inp.write_text("".join(case_text(b, **{k: v for k, v in kw.items()}) for b, kw in cs))
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([str(exe), str(inp)], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    assert "ERROR: AddressSanitizer" not in res.stderr and "runtime error" not in res.stderr, res.stderr[-4000:]
    lines = [l for l in res.stdout.splitlines() if l.startswith("case ")]
    assert len(lines) == len(cs)
    for line, (b, kw) in zip(lines, cs):
        code, stats = library_result(b, kw)
        f = line.split()
        assert int(f[3]) == code, (line, code)
        if code == 0:
            got = (int(f[5]), int(f[7]), int(f[9]), int(f[11]), int(f[13]), int(f[15]))
            assert got == stats, (line, stats)
    assert "allocator free 70" in res.stdout
