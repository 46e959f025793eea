"""A synthetic multi-layer decode step: how much of the time per output token
(TPOT) the attention takes, and what ART's early stop saves end to end.

The paper reports the decode TPOT speedup of ART on whole models (Sec. 4,
Tables 1-2) and explains why it is smaller than the attention speedup and
shrinks with model size (Appendix F): the weight traffic of the projections
and the FFN does not change, and grows faster with parameter count than the
KV cache of a GQA model.  This harness measures that split on one GPU, for
speed only.  Weights are random bf16; each layer's KV cache is a seeded
synthetic cache of the same generator as the attention workloads (its own
seed per layer); there are no trained weights, so there is no quality
measurement.

One step, per layer (batch B, one new token per sequence):
    h = rms_norm(x); qkv = h W_qkv                       (bf16 GEMM)
    a = ART decode attention over the layer's paged cache (bf16 out)
    x = x + a W_o
    h = rms_norm(x); g, u = h W_gate_up; x = x + (silu(g) u) W_down
then rms_norm and the LM head.  The attention consumes the cache's own
query (the workload's q: the synthetic caches are built around it, which is
what makes their early stops representative) and the projected q is left
unused; appending the new token's K and V to the cache is not modelled
(B Hkv 512 bytes per layer).  The step runs eagerly on one stream.

Modes: NODET (full attention, no stability test: the baseline), OFF (test on,
never stops) and ON (the workload thresholds).  Reported per mode: TPOT, the
attention's share, and the speedup over NODET.

    python -m paper_2606_00024_amd.tpot --model llama3_8b --batch 8 --seq-len 32768
"""
from __future__ import annotations

import argparse
import json
import math
import sys
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ModelShape:
    """Decoder shape of one GPU's share (public model cards; head_dim 128)."""
    name: str
    layers: int
    hidden: int
    q_heads: int
    kv_heads: int
    ffn: int
    vocab: int

    def weight_bytes(self) -> int:
        """bf16 weight bytes one decode step reads (projections, FFN, LM head;
        norms and embeddings are negligible)."""
        d = 128
        per_layer = (self.hidden * (self.q_heads + 2 * self.kv_heads) * d
                     + self.q_heads * d * self.hidden
                     + self.hidden * 2 * self.ffn + self.ffn * self.hidden)
        return 2 * (self.layers * per_layer + self.hidden * self.vocab)

    def kv_bytes(self, batch: int, seq_len: int) -> int:
        """bf16 K and V bytes of the whole cache (all layers)."""
        return self.layers * batch * seq_len * self.kv_heads * 128 * 2 * 2


MODELS = {
    # Mistral-7B-v0.3 (the paper's single-GPU model): 32 layers, 4096 hidden,
    # 32/8 heads, FFN 14336, vocabulary 32768
    "mistral_7b": ModelShape("mistral_7b", 32, 4096, 32, 8, 14336, 32768),
    # Llama-3-8B: as above with a 128256-entry vocabulary
    "llama3_8b": ModelShape("llama3_8b", 32, 4096, 32, 8, 14336, 128256),
    # Qwen3-8B: 36 layers, 4096 hidden, 32/8 heads, FFN 12288, vocabulary 151936
    "qwen3_8b": ModelShape("qwen3_8b", 36, 4096, 32, 8, 12288, 151936),
    # Llama-3.1-70B at tensor parallelism 4 (the paper's four-GPU setting), one
    # GPU's share: 80 layers, 8192 hidden, 16/2 heads, FFN 7168, a quarter of
    # the vocabulary (the all-reduces between GPUs are not modelled)
    "llama3_70b_tp4": ModelShape("llama3_70b_tp4", 80, 8192, 16, 2, 7168, 128256 // 4),
}


class Step:
    """Weights, caches and pre-marshalled attention calls of one model."""

    def __init__(self, model: ModelShape, batch: int, seq_len: int, seed: int = 11,
                 tau: float = 1e-3, phi: float = 1e-4, patience: int = 5):
        import torch
        from . import _lib, api, workloads as W
        self.torch = torch
        self._lib = _lib
        self.model, self.batch, self.seq_len = model, batch, seq_len
        dev = torch.device("cuda", torch.cuda.current_device())
        gen = torch.Generator(device=dev).manual_seed(seed)
        d = 128

        def weight(rows, cols):
            w = torch.empty((rows, cols), dtype=torch.bfloat16, device=dev)
            w.normal_(0.0, 1.0 / math.sqrt(rows), generator=gen)
            return w

        m = model
        self.layers = []
        for layer in range(m.layers):
            spec = W.WorkloadSpec(name=f"{m.name}_layer{layer}", batch=batch, num_q_heads=m.q_heads,
                                  num_kv_heads=m.kv_heads, seq_lens=(seq_len,) * batch,
                                  tau=tau, phi=phi, patience=patience, seed=1000 * seed + layer)
            wl = W.make_workload(spec, device=dev)
            self.layers.append({
                "wl": wl,
                "w_qkv": weight(m.hidden, (m.q_heads + 2 * m.kv_heads) * d),
                "w_o": weight(m.q_heads * d, m.hidden),
                "w_gu": weight(m.hidden, 2 * m.ffn),
                "w_d": weight(m.ffn, m.hidden),
            })
        self.w_head = weight(m.hidden, m.vocab)
        self.x0 = torch.empty((batch, m.hidden), dtype=torch.bfloat16, device=dev).normal_(generator=gen)
        self.out = torch.empty((batch, m.q_heads, d), dtype=torch.bfloat16, device=dev)
        self.lse = torch.empty((batch, m.q_heads), dtype=torch.float32, device=dev)
        self.stop = [torch.empty((batch, m.kv_heads), dtype=torch.int32, device=dev)
                     for _ in range(m.layers)]
        self.stream = torch.cuda.current_stream(dev).cuda_stream
        p = lambda t: 0 if t is None else int(t.data_ptr())
        self.calls = {}
        ws_bytes = 0
        for mode, kw in (("nodet", dict(tau=0.0, phi=0.0, patience=1, no_detector=True)),
                         ("off", dict(tau=0.0, phi=phi, patience=patience)),
                         ("on", dict(tau=tau, phi=phi, patience=patience))):
            per_layer = []
            for li, L in enumerate(self.layers):
                wl = L["wl"]
                shape = api.make_shape(wl.q, wl.k_cache, wl.v_cache, wl.page_table,
                                       block_size=wl.spec.block_size)
                opts = api.make_opts(softmax_scale=wl.spec.softmax_scale, out_dtype=torch.bfloat16,
                                     dense_order=wl.spec.dense_order, **kw)
                ws_bytes = max(ws_bytes, api.workspace_bytes(shape, opts))
                per_layer.append((shape, opts, (p(wl.q), p(wl.k_cache), p(wl.v_cache), p(wl.page_table),
                                                p(wl.seq_lens), 0, 0, p(self.out), p(self.lse),
                                                p(self.stop[li]))))
            self.calls[mode] = per_layer
        self.ws = api.new_workspace(ws_bytes, dev)

    def attention(self, mode: str, layer: int):
        shape, opts, args = self.calls[mode][layer]
        st = self._lib.decode_attention(shape, opts, *args, int(self.ws.data_ptr()), self.ws.numel(),
                                        self.stream)
        if st != 0:
            raise self._lib.ArtError(st, "art_decode_attention")
        return self.out

    def run(self, mode: str, attention: bool = True, dense: bool = True):
        """One decode step; `attention` / `dense` switch the two parts off
        (for the split of the time, never for the reported TPOT)."""
        torch = self.torch
        F = torch.nn.functional
        m = self.model
        x = self.x0
        for li, L in enumerate(self.layers):
            if dense:
                h = F.rms_norm(x, (m.hidden,))
                _ = h @ L["w_qkv"]
            if attention:
                a = self.attention(mode, li).view(self.batch, m.q_heads * 128)
            else:
                a = self.out.view(self.batch, m.q_heads * 128)
            if dense:
                x = x + a @ L["w_o"]
                h = F.rms_norm(x, (m.hidden,))
                gu = h @ L["w_gu"]
                g, u = gu.split(m.ffn, dim=1)
                x = x + (F.silu(g) * u) @ L["w_d"]
        if dense:
            _ = F.rms_norm(x, (m.hidden,)) @ self.w_head
        return x

    def time_ms(self, mode: str, steps: int, warmup: int, **kw) -> np.ndarray:
        torch = self.torch
        for _ in range(warmup):
            self.run(mode, **kw)
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(steps)]
        for e0, e1 in evs:
            e0.record()
            self.run(mode, **kw)
            e1.record()
        torch.cuda.synchronize()
        return np.array([e0.elapsed_time(e1) for e0, e1 in evs])

    def skipped_pct(self, mode: str) -> float:
        self.run(mode, dense=False)
        self.torch.cuda.synchronize()
        T = self.seq_len // 64 if self.seq_len % 64 == 0 else -(-self.seq_len // 64)
        total = self.model.layers * self.batch * self.model.kv_heads * T
        consumed = sum(int(s.sum()) for s in self.stop)
        return 100.0 * (1 - consumed / total)


def measure(model: ModelShape, batch: int, seq_len: int, steps: int = 10, warmup: int = 3) -> dict:
    step = Step(model, batch, seq_len)
    res = {"model": model.name, "batch": batch, "seq_len": seq_len, "layers": model.layers,
           "weight_gb": model.weight_bytes() / 1e9, "kv_gb": model.kv_bytes(batch, seq_len) / 1e9,
           "dense_only_ms": float(np.median(step.time_ms("nodet", steps, warmup, attention=False))),
           "modes": {}}
    for mode in ("nodet", "off", "on"):
        tpot = float(np.median(step.time_ms(mode, steps, warmup)))
        attn = float(np.median(step.time_ms(mode, steps, warmup, dense=False)))
        res["modes"][mode] = {"tpot_ms": tpot, "attention_ms": attn,
                              "attention_share": attn / tpot, "skipped_pct": step.skipped_pct(mode)}
    base = res["modes"]["nodet"]
    for mode, r in res["modes"].items():
        r["tpot_speedup_vs_nodet"] = base["tpot_ms"] / r["tpot_ms"]
        r["attention_speedup_vs_nodet"] = base["attention_ms"] / r["attention_ms"]
    return res


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--model", default="llama3_8b", choices=sorted(MODELS))
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--seq-len", type=int, default=32768)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--json", default=None)
    args = ap.parse_args(argv)
    res = measure(MODELS[args.model], args.batch, args.seq_len, steps=args.steps)
    print(json.dumps(res), flush=True)
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
