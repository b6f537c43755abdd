"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI
binding, run the fp64 oracle on the same seeded inputs, compare."""
from __future__ import annotations

import sys
import time

import numpy as np

from oracle import nlr as onlr

U_TOL = 1e-4     # max_ij |U_gpu - U_ref| / max_ij |U_ref| per iteration
OBJ_TOL = 1e-5   # relative error of the objective


_T0 = time.time()


def log(msg: str) -> None:
    print(f"[{time.time() - _T0:7.1f}s] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(a, dtype=np.float32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).to("cuda:0")


def make_ctx(X, Z, K, alpha, beta=1.0, eps_d=1e-4, eps_c=1e-4, T_min=0, flags=0, y0=None, stream=None):
    from paper_2609_36074_amd import nlr
    Xt, Ut = to_dev(X), to_dev(Z)
    yt = None if y0 is None else to_dev(y0)
    ctx = nlr.Context(Xt, K, Ut, yt, alpha=alpha, beta=beta, eps_d=eps_d, eps_c=eps_c, T_min=T_min,
                      flags=flags, stream=stream)
    return ctx


def host(t) -> np.ndarray:
    return t.detach().cpu().numpy().astype(np.float64)


def rel_max_err(a, ref) -> float:
    scale = np.abs(ref).max()
    return float(np.abs(np.asarray(a, np.float64) - ref).max() / (scale if scale > 0 else 1.0))


def obj_rel_err(a: float, ref: float, scale: float) -> float:
    return abs(a - ref) / max(abs(ref), scale)


def label_agreement(lab_gpu: np.ndarray, U_ref: np.ndarray, rel_gap: float = 2e-4):
    """(mismatches on unambiguous rows, number of ambiguous rows).  A row is
    ambiguous when its top-2 gap in the reference is <= rel_gap * its max."""
    srt = np.sort(U_ref, axis=1)
    top = srt[:, -1]
    gap = top - (srt[:, -2] if U_ref.shape[1] > 1 else 0.0)
    amb = gap <= rel_gap * np.maximum(top, 1e-300)
    ref = onlr.labels(U_ref)
    bad = (lab_gpu != ref) & ~amb
    return int(bad.sum()), int(amb.sum())


def trajectory(X, Z, K, alpha, beta, T, eps_d=1e-4, eps_c=1e-4, one_step_tol=None, flags=0):
    """Steps the GPU T times; returns per-iteration errors vs the oracle (gate replay)
    and per-iteration one-step errors (oracle step from the GPU's own iterate)."""
    ctx = make_ctx(X, Z, K, alpha, beta, eps_d=eps_d, eps_c=eps_c, T_min=T, flags=flags)
    Xh, _, _ = onlr.centre_and_normalise(X)
    n = X.shape[0]
    U_gpu = [host(ctx.U)]
    y_gpu = [host(ctx.y)]
    stats = []
    for t in range(T):
        stats.append(ctx.step())
        U_gpu.append(host(ctx.U))
        y_gpu.append(host(ctx.y))
    gates = [bool(s["dual_step"]) for s in stats]
    ref = onlr.run(Xh, Z, K, alpha, beta, T=T, T_min=T, eps_d=eps_d, eps_c=eps_c, gates=gates,
                   keep_trajectory=True)
    traj_err = [rel_max_err(U_gpu[t + 1], ref.trajectory[t]) for t in range(T)]
    obj_err = [obj_rel_err(stats[t]["objective"], ref.records[t].objective, 1.0) for t in range(T)]
    # gate decisions against the oracle's own movement
    bad_gates = [t for t in range(T)
                 if gates[t] != (ref.records[t].delta < eps_d)
                 and abs(ref.records[t].delta - eps_d) > 1e-3 * eps_d]
    one = []
    if one_step_tol is not None:
        for t in range(T):
            y_math = onlr.dual_from_stored(y_gpu[t])
            r1 = onlr.run(Xh, U_gpu[t], K, alpha, beta, T=1, T_min=1, project_init=False, y0=y_math,
                          gates=[gates[t]])
            one.append(rel_max_err(U_gpu[t + 1], r1.U))
            ystored = onlr.stored_dual(r1.y)
            assert np.abs(y_gpu[t + 1] - ystored).max() <= 1e-5 * max(1e-12, np.abs(ystored).max()) + 1e-12, t
    return ctx, ref, traj_err, obj_err, bad_gates, one, U_gpu, stats


def lockstep(ctx, Xh, U0, K, alpha, beta, T, eps_d, t0=0):
    """Steps the GPU context T times (nlr_step with its record) and the fp64 oracle along,
    holding a few copies of U only (no stored trajectory), for the full-size workloads:
      traj[t]  the oracle's own trajectory from U0 (the GPU's gate decisions replayed) at t+1;
      one[t]   one oracle step from the GPU's own iterate U_t, y_t (same gate), at t+1;
      yerr[t]  the stored dual after that step, relative to its max;
      obj[t]   the objective f_{y_t}(U_t) of the record against the trajectory's.
    The oracle steps run one after the other in this thread: BLAS calls made concurrently
    from two Python threads have returned wrong products here."""
    U_ref = np.asarray(U0, dtype=np.float64)
    y_ref = np.zeros(U_ref.shape[0])
    U_prev, y_prev = host(ctx.U), host(ctx.y)
    out = {"traj": [], "one": [], "yerr": [], "obj": [], "bad_gates": [], "stats": []}

    def oracle_step(U, y, gate, t):
        return onlr.run(Xh, U, K, alpha, beta, T=1, T_min=1, project_init=False, y0=y, gates=[gate], t0=t)

    for t in range(t0, t0 + T):
        st = ctx.step()
        out["stats"].append(st)
        gate = bool(st["dual_step"])
        U_gpu, y_gpu = host(ctx.U), host(ctx.y)
        r = oracle_step(U_ref, y_ref, gate, t)
        rec = r.records[0]
        out["traj"].append(rel_max_err(U_gpu, r.U))
        out["obj"].append(obj_rel_err(st["objective"], rec.objective, 1.0))
        if gate != (rec.delta < eps_d) and abs(rec.delta - eps_d) > 1e-3 * eps_d:
            out["bad_gates"].append(t)
        U_ref, y_ref = r.U, r.y
        del r
        o = oracle_step(U_prev, onlr.dual_from_stored(y_prev), gate, t)
        out["one"].append(rel_max_err(U_gpu, o.U))
        ys = onlr.stored_dual(o.y)
        ymax = float(np.abs(ys).max())
        out["yerr"].append(float(np.abs(y_gpu - ys).max()) / ymax if ymax > 0 else float(np.abs(y_gpu).max()))
        del o
        U_prev, y_prev = U_gpu, y_gpu
        log(f"  t={t}: traj {out['traj'][-1]:.2e} one {out['one'][-1]:.2e} obj {out['obj'][-1]:.2e} "
            f"gate {int(gate)}")
    out["U_ref"], out["U_gpu"] = U_ref, U_prev
    return out


# ---------------------------------------------------------------- full-size lockstep in parallel
# The GPU's iterates of a full-size run are saved first (float32, as read back); then one
# worker process runs the oracle's trajectory from U_0 (the GPU's gate decisions
# replayed) and the others run one oracle step from each saved GPU iterate.  The oracle
# steps of a worker run one after another (BLAS in several threads of one process has
# returned wrong products here); the workers are spawned processes that never touch
# the GPU and read Xhat and the iterates from files mapped into memory.

def _scratch_dir(need_bytes: int) -> str:
    import shutil
    import tempfile
    for base in ("/dev/shm", tempfile.gettempdir()):
        try:
            if shutil.disk_usage(base).free > 1.5 * need_bytes:
                return tempfile.mkdtemp(prefix="nlr_lock_", dir=base)
        except OSError:
            continue
    raise RuntimeError(f"no scratch space for {need_bytes / 2**30:.1f} GiB of iterates")


def _load(path: str, dtype=np.float64) -> np.ndarray:
    return np.asarray(np.load(path, mmap_mode="r"), dtype=dtype)


def _blas_threads(threads):
    import threadpoolctl
    return threadpoolctl.threadpool_limits(threads)


def _traj_task(d, K, alpha, beta, gates, eps_d, sources, threads):
    """Oracle trajectory from U_0 with the gates given; per iteration the relative error
    against each source's saved iterate, the objective and the movement; and the label
    agreement of each source's labels with the trajectory at the source's last iteration."""
    _blas_threads(threads)
    Xh = np.load(f"{d}/Xh.npy", mmap_mode="r")
    U = _load(f"{d}/U0.npy")
    y = np.zeros(U.shape[0])
    out = {"err": {s: [] for s, _ in sources}, "obj": [], "delta": [], "labels": {}}
    for t, gate in enumerate(gates):
        r = onlr.run(Xh, U, K, alpha, beta, T=1, T_min=1, project_init=False, y0=y, gates=[gate], t0=t)
        U, y = r.U, r.y
        out["obj"].append(r.records[0].objective)
        out["delta"].append(r.records[0].delta)
        for s, T_s in sources:
            if t < T_s:
                out["err"][s].append(rel_max_err(_load(f"{d}/{s}_U{t + 1}.npy"), U))
            if t + 1 == T_s:  # the source's labels were taken after its last iteration
                out["labels"][s] = label_agreement(np.load(f"{d}/{s}_labels.npy"), U)
        del r
        log(f"    oracle trajectory: iteration {t} done")
    return out


def _one_task(d, K, alpha, beta, src, t, gate, threads):
    """One oracle step from a source's saved iterate t; (U error, stored-dual error) at t+1."""
    _blas_threads(threads)
    Xh = np.load(f"{d}/Xh.npy", mmap_mode="r")
    U_t, y_t = _load(f"{d}/{src}_U{t}.npy"), _load(f"{d}/{src}_y{t}.npy")
    o = onlr.run(Xh, U_t, K, alpha, beta, T=1, T_min=1, project_init=False,
                 y0=onlr.dual_from_stored(y_t), gates=[gate], t0=t)
    del U_t
    err = rel_max_err(_load(f"{d}/{src}_U{t + 1}.npy"), o.U)
    ys = onlr.stored_dual(o.y)
    y1 = _load(f"{d}/{src}_y{t + 1}.npy")
    ymax = float(np.abs(ys).max())
    yerr = float(np.abs(y1 - ys).max()) / ymax if ymax > 0 else float(np.abs(y1).max())
    log(f"    oracle step from {src} iterate {t} done")
    return src, t, err, yerr


def lockstep_parallel(runs, Xh, U0, K, alpha, beta, eps_d, workers=3):
    """runs: {name: (ctx, T)}, contexts started from the same Xhat and U0 = Pi_Omega(Z).
    Steps each context T times (one host call per iteration) saving every iterate, then
    checks them against the oracle as ``lockstep`` does, in `workers` processes:
    traj, one, yerr, obj and bad_gates per run, and the label agreement after its last step."""
    import multiprocessing as mp
    import shutil
    from concurrent.futures import ProcessPoolExecutor

    n, r = U0.shape
    need = Xh.nbytes + U0.nbytes + sum((T + 1) * (n * r * 4 + n * 4) for _, T in runs.values())
    d = _scratch_dir(need)
    try:
        np.save(f"{d}/Xh.npy", Xh)
        np.save(f"{d}/U0.npy", U0)
        res = {}
        for s, (ctx, T) in runs.items():
            np.save(f"{d}/{s}_U0.npy", ctx.U.detach().cpu().numpy())
            np.save(f"{d}/{s}_y0.npy", ctx.y.detach().cpu().numpy())
            stats = []
            for t in range(T):
                stats.append(ctx.step())
                np.save(f"{d}/{s}_U{t + 1}.npy", ctx.U.detach().cpu().numpy())
                np.save(f"{d}/{s}_y{t + 1}.npy", ctx.y.detach().cpu().numpy())
            np.save(f"{d}/{s}_labels.npy", ctx.labels().cpu().numpy())
            res[s] = {"stats": stats, "gates": [bool(x["dual_step"]) for x in stats]}
            log(f"  {s}: {T} GPU iterations saved")
        # one trajectory per gate sequence: a run whose gates are a prefix of an earlier
        # run's shares that run's trajectory
        groups = []  # (gates, [(source, T)])
        for s, (_, T) in runs.items():
            g = res[s]["gates"]
            for gg, members in groups:
                if gg[:len(g)] == g:
                    members.append((s, T))
                    break
            else:
                groups.append((g, [(s, T)]))
        # BLAS threads per worker: the box's share of cores (16) split between the workers
        threads = max(1, 16 // workers)
        with ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn")) as ex:
            fts = [ex.submit(_traj_task, d, K, alpha, beta, gg, eps_d, members, threads) for gg, members in groups]
            fo = [ex.submit(_one_task, d, K, alpha, beta, s, t, res[s]["gates"][t], threads)
                  for s, (_, T) in runs.items() for t in range(T)]
            ones = [f.result() for f in fo]
            trs = [f.result() for f in fts]
        for s, (_, T) in runs.items():
            tr = next(x for x, (_, members) in zip(trs, groups) if any(m == s for m, _ in members))
            o = sorted([x for x in ones if x[0] == s], key=lambda x: x[1])
            st = res[s]["stats"]
            res[s].update(traj=tr["err"][s], one=[x[2] for x in o], yerr=[x[3] for x in o],
                          obj=[obj_rel_err(st[t]["objective"], tr["obj"][t], 1.0) for t in range(T)],
                          bad_gates=[t for t in range(T) if res[s]["gates"][t] != (tr["delta"][t] < eps_d)
                                     and abs(tr["delta"][t] - eps_d) > 1e-3 * eps_d],
                          labels=tr["labels"][s])
            for t in range(T):
                log(f"  {s} t={t}: traj {res[s]['traj'][t]:.2e} one {res[s]['one'][t]:.2e} "
                    f"obj {res[s]['obj'][t]:.2e} y {res[s]['yerr'][t]:.2e} gate {int(res[s]['gates'][t])}")
        return res
    finally:
        shutil.rmtree(d, ignore_errors=True)
