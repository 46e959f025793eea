"""GPU-vs-oracle comparison with the acceptance rule of the parity tests.

* stop_block: bit-exact, except for a group whose oracle trace has, at some
  step t <= max(stop_gpu, stop_oracle), |d_scale - tau| <= 1e-5 or
  |d_direction - phi| <= 1e-5 (a near-tie: both decisions are within fp32
  rounding of the threshold).  Such groups are counted and their out/lse are
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

TIE_BAND = 1e-5
OUT_TOL = 2e-3
LSE_TOL = 1e-4


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

    def __str__(self):
        return (f"groups={self.groups} stop_equal={self.stop_equal} near_ties={len(self.near_ties)} "
                f"max_rel_l2={self.max_rel_l2:.3e} max_lse_err={self.max_lse_err:.3e} "
                f"failures={self.failures[:5]}")


def _rel_l2(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    num = np.linalg.norm(a - b, axis=-1)
    den = np.linalg.norm(b, axis=-1)
    return np.where(den > 0, num / np.maximum(den, 1e-300), num)


def near_tie(trace_g: np.ndarray, upto: int, tau: float, phi: float, tau_rel=None) -> bool:
    """trace_g [steps][g][2] of one group.  The d_scale band is TIE_BAND, or
    tau_rel * tau when given (the accumulator reading, whose d_scale is a
    difference of two accumulators and carries their fp32 error)."""
    t = trace_g[: max(0, upto)]
    if t.size == 0:
        return False
    ds, dr = t[..., 0], t[..., 1]
    tau32, phi32 = float(np.float32(tau)), float(np.float32(phi))
    band = TIE_BAND if tau_rel is None else tau_rel * tau32
    with np.errstate(invalid="ignore"):
        hit = (np.abs(ds - tau32) <= band) | (np.abs(dr - phi32) <= TIE_BAND)
    return bool(np.nan_to_num(hit).any())


def compare_group(rep: Report, tag, out_g, lse_g, stop_g, ref_out, ref_lse, ref_stop, trace_g,
                  tau, phi, rerun, tau_rel=None):
    """One (b, kvh) group.  out_g/ref_out [g][D]; rerun(stop) -> (out, lse)
    of the oracle forced to stop at `stop`."""
    rep.groups += 1
    if stop_g == ref_stop:
        rep.stop_equal += 1
        o_ref, l_ref = ref_out, ref_lse
    else:
        if trace_g is None or not near_tie(trace_g, max(stop_g, ref_stop), tau, phi, tau_rel):
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


def compare_workload(wl, gpu, *, tau, phi, patience, dense_order=None, report=None,
                     num_threads=0, probe_stride=1, scale_of_accumulator=False,
                     tau_rel=None) -> Report:
    """Whole workload (small sizes): oracle on every group."""
    rep = report or Report()
    s = wl.spec
    g = s.group_size
    out, lse, stop = (x.detach().float().cpu().numpy() if x.dtype != torch.int32 else x.cpu().numpy()
                      for x in gpu)
    T = max([max(r) for r in wl.traversal_lengths()] + [1])
    do = s.dense_order if dense_order is None else dense_order
    ref = oracle.decode_workload(wl, tau=tau, phi=phi, patience=patience, dense_order=do,
                                 trace_steps=T, num_threads=num_threads,
                                 probe_stride=probe_stride,
                                 scale_of_accumulator=scale_of_accumulator)
    for b in range(s.batch):
        for h in range(s.num_kv_heads):
            def rerun(st, b=b, h=h):
                fs = np.zeros((s.batch, s.num_kv_heads), dtype=np.int32)
                m = np.zeros((s.batch, s.num_kv_heads), dtype=np.uint8)
                fs[b, h] = st
                m[b, h] = 1
                r = oracle.decode_workload(wl, tau=tau, phi=phi, patience=patience,
                                           dense_order=do, force_stop=fs, group_mask=m,
                                           probe_stride=probe_stride,
                                           scale_of_accumulator=scale_of_accumulator)
                return r["out"][b, h * g:(h + 1) * g], r["lse"][b, h * g:(h + 1) * g]
            compare_group(rep, (b, h), out[b, h * g:(h + 1) * g].astype(np.float64),
                          lse[b, h * g:(h + 1) * g].astype(np.float64), int(stop[b, h]),
                          ref["out"][b, h * g:(h + 1) * g], ref["lse"][b, h * g:(h + 1) * g],
                          int(ref["stop"][b, h]), ref["trace"][b, h], tau, phi, rerun,
                          tau_rel)
    return rep


def compare_sampled(wl, gpu, groups, *, tau, phi, patience, report=None, num_threads=0,
                    probe_stride=1) -> Report:
    """Full-size workloads: the oracle runs on host copies of the sampled
    groups only (workloads.group_subproblem)."""
    from paper_2606_00024_amd.workloads import group_subproblem
    rep = report or Report()
    s = wl.spec
    g = s.group_size
    out, lse, stop = gpu
    for (b, h) in groups:
        sub = group_subproblem(wl, b, h)
        T = max(1, int(sub["block_list_len"][0, 0]) if sub["block_list"] is not None
                else -(-int(sub["seq_lens"][0]) // s.block_size))
        kw = dict(block_size=s.block_size, scale=s.softmax_scale, tau=tau, phi=phi,
                  patience=patience, dense_order=s.dense_order, block_list=sub["block_list"],
                  block_list_len=sub["block_list_len"], num_threads=num_threads,
                  probe_stride=probe_stride)
        ref = oracle.decode(sub["q"], sub["k_cache"], sub["v_cache"], sub["page_table"],
                            sub["seq_lens"], trace_steps=T, **kw)

        def rerun(st, sub=sub, kw=kw):
            r = oracle.decode(sub["q"], sub["k_cache"], sub["v_cache"], sub["page_table"],
                              sub["seq_lens"], force_stop=np.array([[st]], dtype=np.int32), **kw)
            return r["out"][0], r["lse"][0]
        o = out[b, h * g:(h + 1) * g].float().cpu().numpy().astype(np.float64)
        l = lse[b, h * g:(h + 1) * g].cpu().numpy().astype(np.float64)
        compare_group(rep, (b, h), o, l, int(stop[b, h]), ref["out"][0], ref["lse"][0],
                      int(ref["stop"][0, 0]), ref["trace"][0, 0], tau, phi, rerun)
    return rep
