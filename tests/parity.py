"""Shared helpers for GPU parity tests: run a step on the device, recompute it
with the fp64 oracle, and compare to the stated tolerances.

Large workloads are checked by ``OracleChecker``: the oracle runs in a pool
of worker processes (one job per request and KV head, or per request for
sampled rows), reading the step's pools, queries and GPU outputs from
memory-mapped files, and each job reports the error statistics of its rows.
"""

from __future__ import annotations

import atexit
import contextlib
import multiprocessing as mp
import os
import shutil
import tempfile

import numpy as np

import oracle

# Tolerances for bf16 inputs with fp32 accumulation, bf16 output.
MAX_ABS = 1e-2       # every output element
REL_L2 = 2e-2        # ||O_gpu - O_ref||_2 / ||O_ref||_2, per request
LSE_ABS = 1e-2


def compact_ids(batch, pages, allow_missing=False):
    """Relabel page ids as indices into the compact page arrays.  With
    ``allow_missing``, pages the compact arrays do not hold map to entry 0:
    the caller guarantees that no checked row sees a key on them (they hold
    other finite data, which the causal mask then hides)."""
    index = {int(p): i for i, p in enumerate(pages)}
    look = (lambda p: index.get(int(p), 0)) if allow_missing else (lambda p: index[int(p)])
    pp = [np.array([look(p) for p in pl], np.int64) for pl in batch.prefix_pages]
    sp = [np.array([look(p) for p in pl], np.int64) for pl in batch.suffix_pages]
    return pp, sp


def expected_pools(batch, hv):
    """Oracle's pool contents (compact) after the step's append."""
    _, sp = compact_ids(batch, hv.pages)
    return oracle.append_kv(hv.k_pages, hv.v_pages, sp, batch.suffix_len, batch.n_rows, hv.k_new, hv.v_new)


def reference(batch, hv, pools=None, rows=None, scale=None):
    pp, sp = compact_ids(batch, hv.pages)
    kp, vp = pools if pools is not None else expected_pools(batch, hv)
    return oracle.prefix_shared_attention(kp, vp, pp, batch.prefix_len, batch.agent, sp, batch.suffix_len,
                                          batch.n_rows, hv.q, batch.num_q_heads, scale=scale, rows=rows)


def compare(batch, o_bits, lse, o_ref, lse_ref, label=""):
    """Check GPU outputs against the oracle on every row the oracle computed.
    ``lse`` may be None (the call was made without an LSE output).
    Returns (max_abs, worst_rel, max_lse_err)."""
    o = oracle.bf16_bits_to_f64(o_bits)
    have = ~np.isnan(o_ref[:, 0, 0])
    assert have.any(), "no reference rows"
    assert not np.isnan(o[have]).any(), f"{label}: NaN in GPU output"
    err = np.abs(o[have] - o_ref[have])
    max_abs = float(err.max())
    lse_err = 0.0
    if lse is not None:
        assert not np.isnan(lse[have]).any(), f"{label}: NaN in GPU LSE"
        lse_err = float(np.abs(lse[have] - lse_ref[have]).max())
    worst_rel = 0.0
    q_indptr = batch.q_indptr()
    for r in range(len(batch.agent)):
        sl = slice(q_indptr[r], q_indptr[r + 1])
        m = have[sl]
        if not m.any():
            continue
        ref = o_ref[sl][m]
        rel = np.linalg.norm(o[sl][m] - ref) / max(np.linalg.norm(ref), 1e-30)
        worst_rel = max(worst_rel, float(rel))
    assert max_abs <= MAX_ABS, f"{label}: max-abs {max_abs:.3e}"
    assert worst_rel <= REL_L2, f"{label}: relative error {worst_rel:.3e}"
    assert lse_err <= LSE_ABS, f"{label}: LSE error {lse_err:.3e}"
    return max_abs, worst_rel, lse_err


# --------------------------------------------------------------------------- parallel oracle

_BLAS_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "BLIS_NUM_THREADS")


@contextlib.contextmanager
def _one_blas_thread():
    """Worker processes start with one BLAS thread each (they run in parallel)."""
    old = {k: os.environ.get(k) for k in _BLAS_VARS}
    for k in _BLAS_VARS:
        os.environ[k] = "1"
    try:
        yield
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


_MAPS: dict = {}


def _mapped(path):
    a = _MAPS.get(path)
    if a is None:
        if len(_MAPS) > 16:
            _MAPS.clear()
        a = np.load(path, mmap_mode="r")
        _MAPS[path] = a
    return a


def _oracle_job(job):
    """One request's wanted rows on some query heads: the oracle's result
    against the GPU's.  Returns (request, max_abs, sum sq diff, sum sq ref,
    max lse error, rows checked)."""
    desc, paths, r, heads, want, pos = job
    kp, vp = _mapped(paths["k"]), _mapped(paths["v"])
    q, o_gpu = _mapped(paths["q"]), _mapped(paths["o"])
    lse_gpu = _mapped(paths["lse"]) if paths.get("lse") else None
    n = int(desc["n_rows"][r])
    hq, d = q.shape[1], q.shape[2]
    # A one-request batch: the request's own rows, the wanted ones filled in
    # from the compact query file (np.zeros maps untouched pages lazily).
    q_sub = np.zeros((n, hq, d), np.uint16)
    q_sub[want] = q[pos]
    o_ref, l_ref = oracle.prefix_shared_attention(
        kp, vp, desc["prefix_pages"], desc["prefix_len"], [desc["agent"][r]], [desc["suffix_pages"][r]],
        [desc["suffix_len"][r]], [n], q_sub, hq, scale=desc["scale"], rows={0: want}, heads=heads)
    ref = o_ref[want][:, heads]
    got = oracle.bf16_bits_to_f64(np.asarray(o_gpu[pos])[:, heads])
    if np.isnan(got).any():
        return (r, float("nan"), float("nan"), 1.0, float("nan"), len(want))
    diff = got - ref
    lerr = 0.0
    if lse_gpu is not None:
        lg = np.asarray(lse_gpu[pos], np.float64)[:, heads]
        lerr = float(np.max(np.abs(lg - l_ref[want][:, heads]))) if not np.isnan(lg).any() else float("nan")
    return (r, float(np.max(np.abs(diff))), float(np.sum(diff * diff)), float(np.sum(ref * ref)), lerr, len(want))


class OracleChecker:
    """A pool of spawned worker processes running the fp64 oracle (numpy
    only; they never touch the GPU), fed through memory-mapped files."""

    def __init__(self, workers: int | None = None):
        n = workers or max(1, min(16, len(os.sched_getaffinity(0))))
        base = "/dev/shm" if os.path.isdir("/dev/shm") else None
        self.dir = tempfile.mkdtemp(prefix="pfx_parity_", dir=base)
        self.workers = n
        self._count = 0
        with _one_blas_thread():
            self.pool = mp.get_context("spawn").Pool(n)
        atexit.register(self.close)

    def put(self, arr) -> str:
        self._count += 1
        path = os.path.join(self.dir, f"a{self._count}.npy")
        np.save(path, np.ascontiguousarray(arr))
        return path

    def drop(self, *paths):
        for p in paths:
            if p and os.path.exists(p):
                os.remove(p)

    def submit(self, batch, pages, kp, vp, q_rows, o_rows, lse_rows, rows, scale=None, split_heads=True,
               partial_pages=False):
        """Queue the check of ``rows`` (request -> row indices).  kp / vp:
        compact pools holding ``pages``; q_rows / o_rows / lse_rows: the
        queries, GPU outputs and LSEs of the checked rows only, in request
        order then row order (lse_rows may be None).  ``partial_pages``: the
        pools hold only the pages the checked rows see (see compact_ids).
        Returns a handle for ``collect``."""
        pp, sp = compact_ids(batch, pages, allow_missing=partial_pages)
        desc = dict(prefix_pages=pp, prefix_len=[int(x) for x in batch.prefix_len],
                    agent=[int(x) for x in batch.agent], suffix_pages=sp,
                    suffix_len=[int(x) for x in batch.suffix_len], n_rows=[int(x) for x in batch.n_rows],
                    scale=scale)
        paths = dict(k=self.put(kp), v=self.put(vp), q=self.put(q_rows), o=self.put(o_rows),
                     lse=self.put(lse_rows) if lse_rows is not None else None)
        g, hkv, hq = batch.group, batch.num_kv_heads, batch.num_q_heads
        jobs, at = [], 0
        for r in sorted(rows):
            want = [int(i) for i in rows[r]]
            if not want:
                continue
            pos = np.arange(at, at + len(want))
            at += len(want)
            if split_heads:
                for h in range(hkv):
                    jobs.append((desc, paths, r, list(range(h * g, (h + 1) * g)), want, pos))
            else:
                jobs.append((desc, paths, r, list(range(hq)), want, pos))
        assert at == len(q_rows), "row files do not match the rows asked for"
        # Longest first: the jobs of the largest requests start early.
        jobs.sort(key=lambda j: -len(j[4]) * (int(batch.suffix_len[j[2]]) + 1))
        return (self.pool.map_async(_oracle_job, jobs, chunksize=1), paths, batch)

    def collect(self, handle, label):
        """Wait for a submitted check and assert the tolerances; returns
        (max_abs, worst per-request rel-L2, max LSE error, rows)."""
        res, paths, batch = handle
        out = res.get()
        self.drop(*paths.values())
        per = {}
        for r, mx, sd, sr, le, nrows in out:
            acc = per.setdefault(r, [0.0, 0.0, 0.0, 0.0, 0])
            assert not np.isnan(mx), f"{label}: NaN in GPU output of request {r}"
            assert not np.isnan(le), f"{label}: NaN in GPU LSE of request {r}"
            acc[0] = max(acc[0], mx)
            acc[1] += sd
            acc[2] += sr
            acc[3] = max(acc[3], le)
            acc[4] = nrows
        max_abs = max(v[0] for v in per.values())
        rel = max(np.sqrt(v[1]) / max(np.sqrt(v[2]), 1e-30) for v in per.values())
        lse_err = max(v[3] for v in per.values())
        nrows = sum(v[4] for v in per.values())
        assert max_abs <= MAX_ABS, f"{label}: max-abs {max_abs:.3e}"
        assert rel <= REL_L2, f"{label}: relative error {rel:.3e}"
        assert lse_err <= LSE_ABS, f"{label}: LSE error {lse_err:.3e}"
        return max_abs, float(rel), lse_err, nrows

    def close(self):
        if getattr(self, "pool", None) is not None:
            self.pool.terminate()
            self.pool.join()
            self.pool = None
        shutil.rmtree(self.dir, ignore_errors=True)


_CHECKER = None


def checker() -> OracleChecker:
    global _CHECKER
    if _CHECKER is None:
        _CHECKER = OracleChecker()
    return _CHECKER


def all_rows(batch):
    return {r: list(range(int(n))) for r, n in enumerate(batch.n_rows) if int(n) > 0}


def gather_rows(arr, batch, rows):
    """Rows of a [tokens][...] array for ``rows`` (request -> row indices),
    in request order then row order."""
    q_indptr = batch.q_indptr()
    idx = [q_indptr[r] + int(i) for r in sorted(rows) for i in rows[r]]
    return np.asarray(arr)[np.asarray(idx, np.int64)]
