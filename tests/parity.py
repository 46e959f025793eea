"""GPU-vs-oracle comparison with the acceptance rule of the parity tests.

* stop_block: bit-exact, except where the two stops differ only because a
  stability criterion lies within fp32 rounding of its threshold (a
  near-tie).  The rule is exact about which steps may flip: every step of
  the oracle's trajectory (termination off, so that steps past either stop
  are known) is classed as surely stable, surely unstable, or ambiguous,
  where ambiguous means that some head has d_scale within ``band(tau)`` of
  tau or d_direction within ``band(phi)`` of phi and no head is surely
  unstable.  A GPU stop is excused iff the patience counter of Eq. (3),
  replayed over those classes with each ambiguous step free to go either
  way, can stop exactly there.  The band is 1e-3 of the threshold, at least
  1e-7 (fp32 rounding of outputs of norm about one) and never more than the
  acceptance rule's 1e-5.  Excused groups are counted and their out/lse are
  compared with the oracle re-run stopping where the GPU stopped.
* out: max over heads of ||o_gpu - o_ref||_2 / ||o_ref||_2 <= 2e-3 (fp32 out).
* lse: |lse_gpu - lse_ref| <= 1e-4.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

import oracle

TIE_REL = 1e-3       # band relative to the threshold
TIE_ABS_MIN = 1e-7   # floor: fp32 rounding of a difference of unit-size outputs
TIE_ABS_MAX = 1e-5   # never wider than the acceptance rule's absolute band
OUT_TOL = 2e-3
LSE_TOL = 1e-4
NO_STOP = 2 ** 31 - 1   # patience that never fires: the whole trajectory

# near-tie counts of every comparison made in this process, for the summary
# that tests/conftest.py prints at the end of the run
SUMMARY: dict = {}


def tie_band(thr: float, rel=None) -> float:
    """Half-width of the band around a threshold inside which fp32 may
    decide either way.  ``rel`` replaces the capped relative rule (the
    accumulator reading of d_scale, whose size grows with the mass)."""
    thr = float(np.float32(thr))
    if not math.isfinite(thr) or thr <= 0:
        return 0.0
    if rel is not None:
        return rel * thr
    return min(TIE_ABS_MAX, max(TIE_REL * thr, TIE_ABS_MIN))


@dataclass
class Report:
    groups: int = 0
    stop_equal: int = 0
    near_ties: list = field(default_factory=list)
    max_rel_l2: float = 0.0
    max_lse_err: float = 0.0
    failures: list = field(default_factory=list)

    def ok(self) -> bool:
        return not self.failures

    def near_tie_bound(self) -> int:
        """At most one excused group in twenty (and one in any case)."""
        return max(1, self.groups // 20)

    def __str__(self):
        return (f"groups={self.groups} stop_equal={self.stop_equal} near_ties={len(self.near_ties)} "
                f"max_rel_l2={self.max_rel_l2:.3e} max_lse_err={self.max_lse_err:.3e} "
                f"failures={self.failures[:5]} ties={self.near_ties[:3]}")


def record(name: str, rep: Report) -> None:
    """Add a comparison to the run's summary and check the near-tie bound."""
    g, t, n = SUMMARY.get(name, (0, 0, 0))
    SUMMARY[name] = (g + rep.groups, t + len(rep.near_ties), n + 1)
    assert len(rep.near_ties) <= rep.near_tie_bound(), \
        f"{name}: {len(rep.near_ties)} near-ties in {rep.groups} groups: {rep.near_ties[:10]}"


def _rel_l2(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    num = np.linalg.norm(a - b, axis=-1)
    den = np.linalg.norm(b, axis=-1)
    return np.where(den > 0, num / np.maximum(den, 1e-300), num)


def step_classes(trace_g: np.ndarray, T: int, tau: float, phi: float, tau_rel=None) -> np.ndarray:
    """trace_g [steps][g][2] (d_scale, d_direction per head) of one group's
    whole trajectory.  Returns int8 [T]: 1 surely stable, 0 surely unstable,
    2 ambiguous (fp32 rounding may decide either way)."""
    tau32, phi32 = float(np.float32(tau)), float(np.float32(phi))
    bs, br = tie_band(tau, tau_rel), tie_band(phi)
    ds, dr = trace_g[:T, :, 0], trace_g[:T, :, 1]
    with np.errstate(invalid="ignore"):
        head_stable = (ds < tau32 - bs) & (dr < phi32 - br)
        # NaN (a zero vector, step 1) compares false: surely unstable
        head_unstable = ~(ds < tau32 + bs) | ~(dr < phi32 + br)
    stable = head_stable.all(axis=1)
    unstable = head_unstable.any(axis=1)
    return np.where(stable, 1, np.where(unstable, 0, 2)).astype(np.int8)


def reachable_stops(classes: np.ndarray, patience: int) -> set:
    """Every stop_block that Eq. (3)'s counter can produce when each
    ambiguous step may be stable or not (T when it can run to the end)."""
    T = len(classes)
    runs = {0}
    stops = set()
    for t in range(1, T + 1):
        c = int(classes[t - 1])
        nxt = set()
        for r in runs:
            if c != 0:
                if r + 1 >= patience:
                    stops.add(t)
                else:
                    nxt.add(r + 1)
            if c != 1:
                nxt.add(0)
        runs = nxt
        if not runs:
            break
    if runs:
        stops.add(T)
    return stops


def excused(trace_full: np.ndarray, T: int, stop_gpu: int, stop_ref: int, tau, phi, patience,
            tau_rel=None) -> bool:
    """Whether a stop mismatch is a near-tie (see the module docstring)."""
    if T <= 0:
        return False
    reach = reachable_stops(step_classes(trace_full, T, tau, phi, tau_rel), patience)
    assert stop_ref in reach, (stop_ref, sorted(reach)[:20])  # the oracle's own stop
    return stop_gpu in reach


def compare_group(rep: Report, tag, out_g, lse_g, stop_g, ref_out, ref_lse, ref_stop,
                  tau, phi, patience, full_trace, rerun, tau_rel=None):
    """One (b, kvh) group.  out_g/ref_out [g][D]; full_trace() -> (trace
    [T][g][2] of the whole trajectory, T); rerun(stop) -> (out, lse) of the
    oracle forced to stop at `stop`."""
    rep.groups += 1
    if stop_g == ref_stop:
        rep.stop_equal += 1
        o_ref, l_ref = ref_out, ref_lse
    else:
        trace, T = full_trace()
        if not excused(trace, T, stop_g, ref_stop, tau, phi, patience, tau_rel):
            rep.failures.append((tag, "stop", int(stop_g), int(ref_stop)))
            return
        rep.near_ties.append((tag, int(stop_g), int(ref_stop)))
        o_ref, l_ref = rerun(int(stop_g))
    if ref_stop == 0 and stop_g == 0:
        if np.any(out_g != 0) or not np.all(np.isneginf(lse_g)):
            rep.failures.append((tag, "empty"))
        return
    err = float(_rel_l2(out_g, o_ref).max())
    lerr = float(np.abs(lse_g - l_ref).max())
    rep.max_rel_l2 = max(rep.max_rel_l2, err)
    rep.max_lse_err = max(rep.max_lse_err, lerr)
    if not (err <= OUT_TOL) or not np.isfinite(err):
        rep.failures.append((tag, "out", err))
    if not (lerr <= LSE_TOL) or not np.isfinite(lerr):
        rep.failures.append((tag, "lse", lerr))


def host_copy(wl):
    """A copy of a workload whose tensors live on the host (the oracle reads
    them in place; one copy serves every comparison of a workload)."""
    import copy
    h = copy.copy(wl)
    for name in ("q", "k_cache", "v_cache", "page_table", "seq_lens", "block_list",
                 "block_list_len"):
        t = getattr(wl, name)
        if t is not None:
            setattr(h, name, t.detach().cpu().contiguous())
    return h


def compare_workload(wl, gpu, *, tau, phi, patience, dense_order=None, report=None,
                     num_threads=0, probe_stride=1, scale_of_accumulator=False,
                     tau_rel=None, host=None, name=None) -> Report:
    """The oracle on every group of the workload (``host``: a host copy of
    it, made once by the caller for large workloads)."""
    rep = report or Report()
    s = wl.spec
    g = s.group_size
    src = host if host is not None else wl
    out, lse, stop = (x.detach().float().cpu().numpy() if x.dtype != torch.int32 else x.cpu().numpy()
                      for x in gpu)
    lens = np.asarray(wl.traversal_lengths())
    do = s.dense_order if dense_order is None else dense_order
    kw = dict(dense_order=do, num_threads=num_threads, probe_stride=probe_stride,
              scale_of_accumulator=scale_of_accumulator)
    ref = oracle.decode_workload(src, tau=tau, phi=phi, patience=patience, **kw)
    for b in range(s.batch):
        for h in range(s.num_kv_heads):
            T = int(lens[b, h])

            def mask(b=b, h=h):
                m = np.zeros((s.batch, s.num_kv_heads), dtype=np.uint8)
                m[b, h] = 1
                return m

            def full_trace(b=b, h=h, T=T):
                r = oracle.decode_workload(src, tau=tau, phi=phi, patience=NO_STOP,
                                           group_mask=mask(), trace_steps=max(T, 1), **kw)
                return r["trace"][b, h], T

            def rerun(st, b=b, h=h):
                fs = np.zeros((s.batch, s.num_kv_heads), dtype=np.int32)
                fs[b, h] = st
                r = oracle.decode_workload(src, tau=tau, phi=phi, patience=patience,
                                           force_stop=fs, group_mask=mask(), **kw)
                return r["out"][b, h * g:(h + 1) * g], r["lse"][b, h * g:(h + 1) * g]
            compare_group(rep, (b, h), out[b, h * g:(h + 1) * g].astype(np.float64),
                          lse[b, h * g:(h + 1) * g].astype(np.float64), int(stop[b, h]),
                          ref["out"][b, h * g:(h + 1) * g], ref["lse"][b, h * g:(h + 1) * g],
                          int(ref["stop"][b, h]), tau, phi, patience, full_trace, rerun,
                          tau_rel)
    if name is not None:
        record(name, rep)
    return rep


def compare_per_head(wl, gpu, *, tau, phi, patience, host=None, name=None, probe_stride=1,
                     report=None) -> Report:
    """Per-query-head termination (stop_block [B][Hq]: each head's stop):
    every head's stop bit-exact against the oracle's per-head stop, except a
    near-tie of that head alone (its stop reachable by the patience replay
    over its own trajectory with the in-band steps free); out and lse per
    head against the oracle at the head's stop (re-run with that head forced
    to stop where the GPU's did when they differ)."""
    rep = report or Report()
    s = wl.spec
    g = s.group_size
    src = host if host is not None else wl
    out, lse, stop = (x.detach().float().cpu().numpy() if x.dtype != torch.int32 else x.cpu().numpy()
                      for x in gpu)
    lens = np.asarray(wl.traversal_lengths())
    kw = dict(probe_stride=probe_stride, per_head_stop=True)
    ref = oracle.decode_workload(src, tau=tau, phi=phi, patience=patience, **kw)
    for b in range(s.batch):
        for h in range(s.num_kv_heads):
            T = int(lens[b, h])
            mask = np.zeros((s.batch, s.num_kv_heads), dtype=np.uint8)
            mask[b, h] = 1
            trace = None
            for i in range(g):
                q = h * g + i
                rep.groups += 1
                sg, sr = int(stop[b, q]), int(ref["head_stop"][b, q])
                o_r, l_r = ref["out"][b, q], ref["lse"][b, q]
                if sg != sr:
                    if trace is None:
                        trace = oracle.decode_workload(src, tau=tau, phi=phi, patience=NO_STOP,
                                                       group_mask=mask, trace_steps=max(T, 1),
                                                       probe_stride=probe_stride)["trace"][b, h]
                    if not excused(trace[:, i:i + 1], T, sg, sr, tau, phi, patience):
                        rep.failures.append(((b, q), "head stop", sg, sr))
                        continue
                    rep.near_ties.append(((b, q), sg, sr))
                    fs = np.zeros((s.batch, s.num_q_heads), dtype=np.int32)
                    fs[b, q] = sg
                    r = oracle.decode_workload(src, tau=tau, phi=phi, patience=patience,
                                               force_stop=fs, group_mask=mask, **kw)
                    o_r, l_r = r["out"][b, q], r["lse"][b, q]
                else:
                    rep.stop_equal += 1
                if sr == 0 and sg == 0:
                    if np.any(out[b, q] != 0) or not np.isneginf(lse[b, q]):
                        rep.failures.append(((b, q), "empty"))
                    continue
                err = float(_rel_l2(out[b, q][None].astype(np.float64), o_r[None])[0])
                lerr = abs(float(lse[b, q]) - float(l_r))
                rep.max_rel_l2 = max(rep.max_rel_l2, err)
                rep.max_lse_err = max(rep.max_lse_err, lerr)
                if not (err <= OUT_TOL):
                    rep.failures.append(((b, q), "out", err))
                if not (lerr <= LSE_TOL):
                    rep.failures.append(((b, q), "lse", lerr))
    if name is not None:
        record(name, rep)
    return rep
