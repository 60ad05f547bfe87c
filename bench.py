#!/usr/bin/env python3
"""LoopSpec decode benchmark on one MI355X.

Workload (the headline configuration): the Raven/Huginn-shaped looped decoder
(2 prelude blocks, 4 core blocks iterated R = 32 times, 2 coda blocks; hidden
5280, 55 heads x 96, SwiGLU FFN 17920, vocabulary 65536, bf16, random
N(0, 0.02) weights with residual scale alpha = 0.3), a 1024-token uniform
prompt, greedy decoding of 256 tokens, batch 1, proposal depths
(d1, d2) = (16, 24), the fastest pair of this configuration's grid
(`--sweep raven` measures every pair against vanilla).  `--model ouro14 --d1 2
--d2 3 --prompt 512` gives the Ouro-1.4B-shaped configuration, `--model ouro26
--d1 1 --d2 2 --prompt 1024 --temperature 1 --top-p 0.95` the sampled
Ouro-2.6B-shaped one.

One bench step = rewind to the post-prefill state and decode 256 tokens with
LoopSpec (every step of the hot path: batched recurrence, readouts, drafting,
gating, verification, re-rooting, KV commit, embedding), replaying the
captured step graphs.  Prefill is not timed (the paper times the decode phase
only).  The same decode on the vanilla schedule (all R depths per token) runs
on the same kernels for the speedup.

Roofline: the dominant kernel of the decode -- the persistent pass of the
shared block stack where the model fits it, else the gate/up GEMM of the core
blocks (the largest weight stream) -- measured inside the decode itself: one
more decode of the same tokens launches each step's kernels directly with HIP
events around every launch of that kernel, and each launch's algorithmic bytes
come from the rows of its own step (the weights it streams, the key/value
positions its rows read, their writes).  Also reported: the same kernel in a
synthetic replay (labelled best case), the plain HBM read ceiling, and the
fp64 CPU oracle's vanilla decode on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/s (batch 1) + speedup vs vanilla loop; weight-stream HBM GB/s"
PEAK_HBM_GBS = 8000.0

# HBM bytes of one k_pass launch at the roofline workload (Ouro-1.4B shape,
# M = 2 rows at position 512): rocprofv3 FETCH_SIZE + WRITE_SIZE, each scaled
# by what the counter reads for a plain 1 GiB copy.  Valid only for the
# kernel sources it was measured on (their SHA-1 below); otherwise null.
PASS_TRAFFIC = {"sources_sha1": "e005b90bbe8453e0f70a403a8508c4e045e9d006", "model": "ouro14", "M": 2,
                "pos": 512, "bytes": 2697531611}
PASS_SOURCES = ["ls_common.h", "ls_gemm.h", "ls_gemm_dev.h", "ls_attn.h", "ls_attn_dev.h", "ls_pass.h",
                "ls_pass.hip"]


# HBM bytes of one core-block gate/up launch of the Raven-shaped model at
# M = 2 rows (bench.py --counters: FETCH_SIZE + WRITE_SIZE per dispatch,
# scaled like PASS_TRAFFIC); valid only for the GEMM sources it was measured on
GU_TRAFFIC = {"sources_sha1": "98c6daed010e0b8f4ba6e781ecd77a667a1e5647", "model": "raven", "M": 2,
              "bytes": 379825706}
GEMM_SOURCES = ["ls_common.h", "ls_gemm.h", "ls_gemm_dev.h", "ls_gemm_sk.hip"]

KERNEL_NAME = {
    "pass": "k_pass: persistent decode pass of the shared block stack",
    "gate_up": "k_gemm_sk<SWIGLU>: RMSNorm + gate/up + SwiGLU of a core block (stream-K weight stream, "
               "<= 16 rows)",
}


def gemm_sources_sha1() -> str:
    import hashlib
    hs = hashlib.sha1()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_17184_amd", "csrc", f), "rb") as fh:
            hs.update(fh.read())
    return hs.hexdigest()


def launch_bytes(spec, kind: str, M: int, kvpos: int) -> int:
    """Algorithmic HBM bytes of one launch: the weights it streams once, the
    key/value positions its rows read (each once), and its activations in and
    out (16-bit models compute in fp16: 2-byte activations and caches)."""
    wb = 2 if spec.weight_dtype == "bf16" else 4
    ab = wb
    h, F, L, V = spec.hidden, spec.ffn, spec.n_core, spec.vocab
    if kind == "pass":
        return L * (4 * h * h + 3 * F * h) * wb + L * 2 * h * wb * (kvpos + M) + M * h * 4 * 2
    if kind == "gate_up":
        return 2 * F * h * wb + M * h * ab + M * F * ab + M * (h // 16) * 4
    if kind == "qkv":
        return 3 * h * h * wb + M * h * ab + M * h * 4 + M * 2 * h * wb
    if kind == "o_proj":
        return h * h * wb + M * h * ab + 2 * M * h * 4 + M * h * ab
    if kind == "down":
        return h * F * wb + M * F * ab + 2 * M * h * 4 + M * h * ab
    if kind == "attention":
        return kvpos * 2 * h * wb + M * h * (4 + ab)
    if kind == "head":
        return V * h * wb + M * h * ab + M * V * 4
    raise ValueError(kind)


# depth / residual-scale grids (greedy, batch 1)
SWEEPS = {
    "ouro14": {"alphas": [0.1, 0.3, 0.6], "depths": [(1, 2), (1, 3), (2, 3), (1, 0), (2, 0), (3, 0)],
               "prompt": 512, "tokens": 256},
    "raven": {"alphas": [0.3], "depths": [(4, 8), (4, 12), (8, 12), (8, 16), (16, 20), (16, 24)],
              "prompt": 1024, "tokens": 256},
}


def pass_sources_sha1() -> str:
    import hashlib
    h = hashlib.sha1()
    for f in PASS_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_17184_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--model", default="raven")
    ap.add_argument("--alpha", type=float, default=0.3)
    ap.add_argument("--depths", choices=["fixed", "auto"], default="fixed",
                    help="auto: plan (d1, d2) from the model's teacher-forced readouts along the prompt "
                         "(TV per depth under the run's temperature / top-p, power-law envelope, Theorem 2's "
                         "bound minimised over integer pairs) before decoding")
    ap.add_argument("--d1", type=int, default=16)
    ap.add_argument("--d2", type=int, default=24)
    ap.add_argument("--prompt", type=int, default=1024)
    ap.add_argument("--tokens", type=int, default=256)
    ap.add_argument("--seqs", type=int, default=1)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-tokens", type=int, default=64)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (HBM counter calibration)")
    ap.add_argument("--no-vanilla", action="store_true")
    ap.add_argument("--shared-prefix", action="store_true",
                    help="decode attention of per-kernel handles as shared-prefix tasks (loopspec_config.shared_prefix)")
    ap.add_argument("--counters", action="store_true",
                    help="only the prefill and the best-case pass replay (M = --pass-m, default 2), for "
                         "rocprofv3 --pmc runs, whose counter collection cannot follow graph replays")
    ap.add_argument("--pass-m", type=int, default=0,
                    help="rows of the roofline pass timing (default: the mean effective batch of the timed decode)")
    ap.add_argument("--temperature", type=float, default=0.0, help="0: greedy")
    ap.add_argument("--top-p", type=float, default=1.0)
    ap.add_argument("--seed", type=int, default=2, help="Philox key of the sampling draws")
    ap.add_argument("--second-proposal", type=int, default=0, choices=[0, 1, 2],
                    help="0 gated residual (the method), 1 ungated residual, 2 ungated non-residual (both masked)")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the bench line: the three second-proposal variants under sampling "
                         "(temperature 1, top-p 0.7), LoopSpec vs vanilla, one JSON line each")
    ap.add_argument("--sweep", choices=sorted(SWEEPS), default=None,
                    help="instead of the bench line: LoopSpec vs vanilla over the depth / alpha grid of a "
                         "model, one JSON line per configuration")
    return ap.parse_args()


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(spec, weights, prompt, n_tok, n_prompt=8, r_sample=2):
    """The fp64 oracle's vanilla greedy decode, on a bounded sample.

    The oracle streams fp64 copies of the weights (8 bytes per parameter),
    so the full model is sampled: the same decoder reduced to its first core
    block applied r_sample times, without prelude and coda blocks (the same
    weights for that block, the same widths and LM head), after an untimed
    prefill of the first n_prompt prompt tokens; per generated token the timed
    work is r_sample block applications (LoopedLM.extend) and the LM-head
    readout (LoopedLM.logits).  Every block of the model has the same widths,
    so the full model's time per token is R * n_core + n_prelude + n_coda
    block applications plus one readout."""
    import dataclasses
    from oracle import loopspec as OL
    from oracle import model as OM
    sub = dataclasses.replace(spec, n_prelude=0, n_core=1, n_coda=0, R=r_sample)
    lm = OM.LoopedLM(sub, weights)
    prov = OL.ModelReadouts(lm, prompt[:n_prompt])
    node = prov.root()                              # prefill + weight conversion, not timed
    tok = int(np.argmax(lm.logits(node, sub.R)))    # converts the head, not timed
    t_ext = t_head = 0.0
    for _ in range(n_tok):
        t0 = time.perf_counter()
        node = lm.extend(node, tok)
        t1 = time.perf_counter()
        z = lm.logits(node, sub.R)
        t2 = time.perf_counter()
        t_ext += t1 - t0
        t_head += t2 - t1
        tok = int(np.argmax(z))
    blocks = spec.R * spec.n_core + spec.n_prelude + spec.n_coda
    per_tok = (t_ext / r_sample * blocks + t_head) / n_tok
    try:
        cores = len(os.sched_getaffinity(0))
    except Exception:   # pragma: no cover
        cores = os.cpu_count() or 1
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] + [1])
    except Exception:
        pass
    return {"value": 1.0 / per_tok, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "cpu": cpu_model(),
            "sample": f"fp64 numpy oracle, vanilla greedy decode of {n_tok} tokens through one core block "
                      f"applied {r_sample} times plus the LM-head readout, after an untimed "
                      f"{len(prompt[:n_prompt])}-token prefill; block time scaled to the model's "
                      f"{blocks} block applications per token (R={spec.R} x {spec.n_core} core + "
                      f"{spec.n_prelude} prelude + {spec.n_coda} coda; timed {t_ext + t_head:.1f} s)"}


def sweep(a):
    """LoopSpec vs vanilla over a model's (alpha, d1, d2) grid: one JSON line each."""
    import torch
    import synth
    from paper_2609_17184_amd import Decoder
    g = SWEEPS[a.sweep]
    rows = []
    for alpha in g["alphas"]:
        spec = synth.preset(a.sweep, alpha=alpha)
        weights = synth.make_weights(spec, seed=0)
        prompt = synth.make_prompt(spec.vocab, g["prompt"], seed=1, seq=0)
        max_ctx = g["prompt"] + g["tokens"] + spec.R + 8
        for d1, d2 in g["depths"]:
            dec = Decoder(spec, weights, R=spec.R, d1=d1, d2=d2, max_ctx=max_ctx)
            dec.prefill(0, prompt)
            dec.vanilla_decode(g["tokens"])                  # warm-up (same handle, same kernels)
            dec.rewind(0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            ref = dec.vanilla_decode(g["tokens"])
            torch.cuda.synchronize()
            vanilla = g["tokens"] / (time.perf_counter() - t0)
            dec.rewind(0)
            dec.decode(g["tokens"])                          # warm-up
            dec.rewind(0)
            dec.reset_stats()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            out = dec.decode(g["tokens"])
            torch.cuda.synchronize()
            ls = g["tokens"] / (time.perf_counter() - t0)
            st = dec.stats()
            n = max(1, st["committed"])
            cost = st["n_acc1"] * d1 + st["n_acc2"] * (d2 or spec.R) + st["n_restart"] * spec.R
            row = {"model": a.sweep, "alpha": alpha, "d1": d1, "d2": d2, "tokens_per_s": round(ls, 2),
                   "vanilla_tokens_per_s": round(vanilla, 2), "speedup": round(ls / vanilla, 4),
                   "gamma": round(st["committed"] * spec.R / cost, 4) if cost else None,
                   "first": round(st["n_acc1"] / n, 4), "second": round(st["n_acc2"] / n, 4),
                   "restart": round(st["n_restart"] / n, 4),
                   "gate_open_rate": round(st["gate_open"] / st["gate_eval"], 4) if st["gate_eval"] else None,
                   "mean_M": round(st["sum_M"] / max(1, st["steps"]), 3), "max_M": st["max_M"],
                   "slots": dec.capacity()[0], "pass_kernel": dec.pass_kernel,
                   "identical_to_vanilla": bool(np.array_equal(out, ref))}
            rows.append(row)
            print(json.dumps(row), flush=True)
            dec.close()
    best = max(rows, key=lambda r: r["speedup"])
    print(json.dumps({"sweep": a.sweep, "best": {k: best[k] for k in ("alpha", "d1", "d2", "speedup")}}),
          flush=True)


def ablation(a):
    """Second-proposal variants (Ablation Study, Table 3) on the Ouro-1.4B shape
    under the paper's ablation sampling setting (temperature 1, top-p 0.7)."""
    import torch
    import synth
    from paper_2609_17184_amd import Decoder
    spec = synth.preset(a.model, alpha=a.alpha)
    weights = synth.make_weights(spec, seed=0)
    prompt = synth.make_prompt(spec.vocab, a.prompt, seed=1, seq=0)
    names = {0: "gated residual", 1: "ungated residual, masked", 2: "ungated non-residual, masked"}
    vanilla = None
    for v in (2, 1, 0):
        dec = Decoder(spec, weights, R=spec.R, d1=a.d1, d2=a.d2, temperature=1.0, top_p=0.7, seed=a.seed,
                      max_ctx=a.prompt + a.tokens + spec.R + 8, second_proposal=v)
        dec.prefill(0, prompt)
        if vanilla is None:
            dec.vanilla_decode(a.tokens)
            dec.rewind(0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            dec.vanilla_decode(a.tokens)
            torch.cuda.synchronize()
            vanilla = a.tokens / (time.perf_counter() - t0)
            dec.rewind(0)
        dec.decode(a.tokens)
        rate = []
        st = None
        for it in range(3):                      # three draws of the sampling key
            dec.set_seed(a.seed + 100 * it)
            dec.rewind(0)
            dec.reset_stats()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            dec.decode(a.tokens)
            torch.cuda.synchronize()
            rate.append(a.tokens / (time.perf_counter() - t0))
            s2 = dec.stats()
            st = s2 if st is None else {k: st[k] + s2[k] for k in ("committed", "n_acc1", "n_acc2", "n_restart",
                                                                   "gate_eval", "gate_open", "sum_M", "steps")}
        n = max(1, st["committed"])
        cost = st["n_acc1"] * a.d1 + st["n_acc2"] * a.d2 + st["n_restart"] * spec.R
        ls = float(np.mean(rate))
        print(json.dumps({"ablation": names[v], "second_proposal": v, "model": a.model, "d1": a.d1, "d2": a.d2,
                          "temperature": 1.0, "top_p": 0.7, "tokens_per_s": round(ls, 2),
                          "vanilla_tokens_per_s": round(vanilla, 2), "speedup": round(ls / vanilla, 4),
                          "gamma": round(st["committed"] * spec.R / cost, 4) if cost else None,
                          "first": round(st["n_acc1"] / n, 4), "second": round(st["n_acc2"] / n, 4),
                          "restart": round(st["n_restart"] / n, 4),
                          "second_proposal_rate": round(st["gate_open"] / max(1, st["gate_eval"]), 4),
                          "mean_M": round(st["sum_M"] / max(1, st["steps"]), 3)}), flush=True)
        dec.close()


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {a.gpus}); the path is single-GPU by design",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if a.calibrate_copy:
        n = 1 << 28                                   # 256 Mi fp32 = 1 GiB
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes_read": n * 4, "calibrate_copy_bytes_written": n * 4,
                          "reps": 3}), flush=True)
        return
    import synth
    from paper_2609_17184_amd import Decoder
    if a.sweep:
        return sweep(a)
    if a.ablation:
        return ablation(a)

    spec = synth.preset(a.model, alpha=a.alpha)
    R = spec.R
    t0 = time.time()
    weights = synth.make_weights(spec, seed=0)
    print(f"[bench] weights {spec.n_params() / 1e9:.2f}B params in {time.time() - t0:.1f}s", flush=True)
    prompts = [synth.make_prompt(spec.vocab, a.prompt, seed=1, seq=q) for q in range(a.seqs)]
    max_ctx = a.prompt + a.tokens + R + 8
    plan = None
    if a.depths == "auto":
        from paper_2609_17184_amd import depths as PD
        k0 = min(16, a.prompt // 2)
        pdec = Decoder(spec, weights, R=R, d1=1, d2=2, max_ctx=max_ctx)
        pdec.prefill(0, prompts[0][:k0])
        t0 = time.time()
        plan = PD.select_depths(pdec, 0, prompts[0][k0:k0 + 64], a.temperature, a.top_p)
        pdec.close()
        a.d1, a.d2 = plan["d1"], plan["d2"]
        print(f"[bench] depth plan ({time.time() - t0:.1f}s): TV {plan['tv']}, envelope alpha "
              f"{plan['alpha']:.3f} beta {plan['beta']:.3f}, closed form {plan['closed_form']} "
              f"(valid {plan['closed_form_valid']}), integer argmin ({a.d1}, {a.d2})", flush=True)
    dec = Decoder(spec, weights, R=R, d1=a.d1, d2=a.d2, temperature=a.temperature, top_p=a.top_p,
                  seed=a.seed, max_seqs=a.seqs, max_ctx=max_ctx, second_proposal=a.second_proposal,
                  shared_prefix=a.shared_prefix)
    t0 = time.time()
    for q in range(a.seqs):
        dec.prefill(q, prompts[q])
    torch.cuda.synchronize()
    print(f"[bench] prefill {a.seqs}x{a.prompt} in {time.time() - t0:.2f}s", flush=True)
    if a.counters:
        M = a.pass_m or 2
        ms_pass, fused = dec.time_pass(M, reps=10)
        print(json.dumps({"counters_replay": {"M": M, "reps": 10, "ms": ms_pass, "persistent": bool(fused)}}),
              flush=True)
        dec.close()
        return

    def step():
        for q in range(a.seqs):
            dec.rewind(q)
        return dec.decode(a.tokens)

    for _ in range(a.warmup):
        step()
    dec.reset_stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        out = step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = dec.stats()
    ms_step = dt * 1e3 / a.steps
    value = a.seqs * a.tokens * a.steps / dt
    print(f"[bench] loopspec {value:.1f} tok/s ({ms_step:.1f} ms per {a.tokens}-token decode)", flush=True)

    vanilla = None
    same = None
    if not a.no_vanilla:
        for q in range(a.seqs):
            dec.rewind(q)
        dec.vanilla_decode(a.tokens)                         # warm-up
        t0 = time.perf_counter()
        for q in range(a.seqs):
            dec.rewind(q)
        ref = dec.vanilla_decode(a.tokens)
        torch.cuda.synchronize()
        vdt = time.perf_counter() - t0
        vanilla = a.seqs * a.tokens / vdt
        same = bool(np.array_equal(ref, out)) if a.temperature == 0.0 else None
        print(f"[bench] vanilla {vanilla:.1f} tok/s; identical tokens: {same}", flush=True)

    # roofline of the dominant kernel, inside a decode of the same tokens: HIP
    # events around each of its launches, each launch's bytes from its own rows
    wb = 2 if spec.weight_dtype == "bf16" else 4
    h, F, Lb = spec.hidden, spec.ffn, spec.n_core
    kind = "pass" if dec.pass_kernel else "gate_up"
    for q in range(a.seqs):
        dec.rewind(q)
    prof_ms, prof_info = dec.decode_profile(a.tokens, kind)
    prof_bytes = np.array([launch_bytes(spec, kind, int(m), int(kv)) for m, kv, _ in prof_info], np.float64)
    achieved = float(prof_bytes.sum() / (prof_ms.astype(np.float64).sum() * 1e-3) / 1e9)
    mean_ms = float(prof_ms.mean())
    mean_bytes = float(prof_bytes.mean())
    traffic = None
    if kind == "pass" and pass_sources_sha1() == PASS_TRAFFIC["sources_sha1"] and a.model == PASS_TRAFFIC["model"]:
        traffic = PASS_TRAFFIC["bytes"]
    slots = dec.capacity()[0]
    kname = KERNEL_NAME[kind]
    if kind == "gate_up" and slots > 16:
        # launches of up to 64 rows: stream-K from 64 MB of weights, else the 64-row tiles
        kname = ("k_gemm_sk<SWIGLU, 32 or 64 rows>: RMSNorm + gate/up + SwiGLU of a core block (stream-K weight "
                 "stream, row tiles per wave)" if 2 * F * h * wb >= (64 << 20) else
                 "k_gemm<SWIGLU, 64 rows>: RMSNorm + gate/up + SwiGLU of a core block (64-row LDS tiles)")
    if (kind == "gate_up" and slots <= 16 and gemm_sources_sha1() == GU_TRAFFIC["sources_sha1"]
            and a.model == GU_TRAFFIC["model"]):
        traffic = GU_TRAFFIC["bytes"]
    print(f"[bench] {kname}: {len(prof_ms)} launches in the decode, {mean_ms * 1e3:.1f} us and "
          f"{mean_bytes / 1e6:.1f} MB per launch on average (M {prof_info[:, 0].mean():.2f}): {achieved:.0f} GB/s",
          flush=True)
    # the same pass in a synthetic replay at the mean effective batch (best case:
    # every row at the prompt's end, no in-flight ancestors)
    M = a.pass_m or max(1, int(round(st["sum_M"] / max(1, st["steps"]))))
    for q in range(a.seqs):
        dec.rewind(q)
    ms_pass, fused = dec.time_pass(M, reps=10)
    pos = a.prompt
    replay_bytes = Lb * (4 * h * h + 3 * F * h) * wb + Lb * (min(M, R) * (pos + 1) + M) * 2 * h * wb
    replay_gbs = replay_bytes / (ms_pass * 1e-3) / 1e9
    print(f"[bench] best case: core pass {ms_pass:.4f} ms at M={M} in a replay "
          f"({'persistent kernel' if fused else 'per-kernel launches'}): {replay_gbs:.0f} GB/s", flush=True)
    for q in range(a.seqs):
        dec.rewind(q)
    km = dec.time_kernels(M, reps=3)
    per_kernel_gbs = {
        "qkv": (3 * h * h * wb) / (km["qkv"] * 1e-3) / 1e9,
        "o_proj": (h * h * wb) / (km["o_proj"] * 1e-3) / 1e9,
        "gate_up": (2 * F * h * wb) / (km["gate_up"] * 1e-3) / 1e9,
        "down": (h * F * wb) / (km["down"] * 1e-3) / 1e9,
    }
    print(f"[bench] standalone kernel ms {json.dumps({k: round(v, 4) for k, v in km.items()})} at M={M}",
          flush=True)
    # the practical ceiling of a weight stream: a plain read of 2 GiB
    from paper_2609_17184_amd.binding import read_bandwidth
    probe = torch.ones(1 << 31, dtype=torch.uint8, device="cuda")
    read_ceiling, _ = read_bandwidth(probe, reps=10)
    del probe
    print(f"[bench] plain read stream {read_ceiling:.0f} GB/s; the kernel reaches {achieved / read_ceiling:.3f} of it",
          flush=True)

    cpu = None
    if not a.no_cpu:
        cpu = cpu_baseline(spec, weights, prompts[0], a.cpu_tokens)
        print(f"[bench] cpu oracle {cpu['value']:.3f} tok/s on {cpu['cores']} threads", flush=True)

    decoding = ("greedy decode" if a.temperature == 0.0 else
                f"sampled decode (temperature {a.temperature}, top-p {a.top_p}, speculative rejection, Philox)")
    n_dec = max(1, st["committed"])
    gamma = (st["committed"] * R / (st["n_acc1"] * a.d1 + st["n_acc2"] * (a.d2 or R) + st["n_restart"] * R)
             if st["committed"] else None)
    line = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16" if spec.weight_dtype == "bf16" else "f32",
        "weights_dtype": spec.weight_dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{a.model}-shaped looped decoder ({spec.n_prelude} prelude + {spec.n_core} core blocks "
                        f"x R={R} + {spec.n_coda} coda, h={spec.hidden}, {spec.n_heads}x{spec.head_dim}, "
                        f"F={spec.ffn}, V={spec.vocab}, alpha={a.alpha}), {a.seqs}x{a.prompt}-token prompt, "
                        f"{decoding} of {a.tokens} tokens, (d1,d2)=({a.d1},{a.d2})"
                        + (", shared-prefix attention" if a.shared_prefix else ""),
            "global_batch": a.seqs, "seq_len": a.prompt + a.tokens, "parallelism": "single-gpu",
        },
        "speedup_vs_vanilla": round(value / vanilla, 4) if vanilla else None,
        "vanilla_tokens_per_s": round(vanilla, 3) if vanilla else None,
        "greedy_identical_to_vanilla": same,
        "acceptance": {
            "first": st["n_acc1"] / n_dec, "second": st["n_acc2"] / n_dec, "restart": st["n_restart"] / n_dec,
            "gate_open_rate": (st["gate_open"] / st["gate_eval"]) if st["gate_eval"] else None,
            "gamma": gamma, "mean_M": st["sum_M"] / max(1, st["steps"]), "max_M": st["max_M"],
        },
        "standalone_kernel_ms": {k: round(v, 5) for k, v in km.items()},
        "standalone_kernel_weight_GBps": {k: round(v, 1) for k, v in per_kernel_gbs.items()},
        "roofline": {
            "bound": "hbm",
            "kernel": kname,
            "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
            "measured": f"HIP events carried by the dispatch of each of the {len(prof_ms)} launches of this kernel in a decode of "
                        f"the same {a.tokens} tokens (steps launched directly instead of from the step graph); "
                        f"bytes per launch from that launch's own rows",
            "launches": int(len(prof_ms)), "ms_per_launch": round(mean_ms, 5),
            "bytes_per_launch": round(mean_bytes), "mean_M": round(float(prof_info[:, 0].mean()), 3),
            "read_stream_GBps": round(read_ceiling, 1), "frac_of_read_stream": round(achieved / read_ceiling, 4),
            "best_case": {"what": "core-stack pass replayed with M rows at the prompt's end, no in-flight "
                                  "ancestors", "M": M, "ms": round(ms_pass, 5),
                          "GBps": round(replay_gbs, 1), "frac": round(replay_gbs / PEAK_HBM_GBS, 4)},
        },
        "cpu_baseline": cpu,
    }
    if plan is not None:
        line["depth_plan"] = {"tv": {str(k): round(v, 4) for k, v in plan["tv"].items()},
                              "alpha": round(plan["alpha"], 4), "beta": round(plan["beta"], 4),
                              "closed_form": [round(x, 3) for x in plan["closed_form"]],
                              "closed_form_valid": plan["closed_form_valid"],
                              "d1": plan["d1"], "d2": plan["d2"], "steps_bound": round(plan["steps_bound"], 4)}
    print(json.dumps(line), flush=True)
    dec.close()


if __name__ == "__main__":
    main()
