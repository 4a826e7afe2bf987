"""Throughput of the CORA-Diff denoising step on one MI355X.

A step is one executed denoising pass over one batch: the dense bidirectional pass at
the LLaDA-8B shape (32 layers, d 4096, 32 x 128 heads, SwiGLU 12288, vocab 126464), the
LM head on the active block rows, and the fused vocab/gate kernel (top-1, confidence,
persistence, transfer rule, residual gate, commit, termination).  Workload: batch 1,
prompt 256 seeded random tokens + 256 generated positions, block 32, 32 steps per block,
gate (0.65, 1), seeded N(0, 0.02) bf16 weights.

Prints one JSON line.  value = denoising passes/s; also generated tokens/s, the
roofline of the dominant kernel (gate/up SwiGLU GEMM, timed live with HIP events on the
launching stream), the vocab/gate kernel's HBM roofline on bf16 logits [8, 512, 126464],
a full gated block decode (passes per block, step ratio) and the CPU oracle baseline.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import hashlib

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
B, P, G, BLK, S = 1, 256, 256, 32, 32
DELTA_P, M_REQ = 0.65, 1
TIME_EVERY = 4              # gate/up event timing on every 4th timed pass


# HBM bytes per launch from rocprofv3 FETCH_SIZE (x2.0) + WRITE_SIZE (x1.0) runs, scaled by a
# plain 1 GiB copy (profiles/gate_up_gemm_llada8b_gen256.md, profiles/vocab_gate_8x512x126464.md).
# Valid only for the kernel source the counters were taken on: the digest covers the kernel's
# file and the shared device headers.
SHARED_SOURCES = ("paper_2608_11235_amd/csrc/common.hpp", "paper_2608_11235_amd/csrc/internal.hpp")
COUNTER_TRAFFIC = {
    "gate_up": ("paper_2608_11235_amd/csrc/gemm.hip", "e6476cbe77e4bdc7", 247638118),
    "vocab_gate": ("paper_2608_11235_amd/csrc/vocab_gate.hip", "8158577e35d7c498", 1036529255),
}


def source_digest(path):
    h = hashlib.sha256()
    for p in (path,) + SHARED_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def note(msg):
    """Progress line on stderr (stdout carries the one JSON result line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def counter_traffic(name):
    path, digest, nbytes = COUNTER_TRAFFIC[name]
    return nbytes if digest is not None and source_digest(path) == digest else None


def pass_flops(spec, M, rows, batch=B):
    """Algorithmic FLOPs of one dense pass: GEMMs + attention + LM head on `rows` rows."""
    d, H, Hkv, hd, F, V = (spec.d_model, spec.n_heads, spec.n_kv_heads, spec.head_dim,
                           spec.ffn_dim, spec.vocab)
    L = M // batch
    per_layer = 2 * M * d * (H + 2 * Hkv) * hd + 2 * M * H * hd * d + 2 * M * d * 2 * F \
        + 2 * M * F * d + 4 * batch * H * L * L * hd
    return spec.n_layers * per_layer + 2 * rows * d * V


def gu_flops(spec, M):
    return 2 * M * spec.d_model * 2 * spec.ffn_dim


def cpu_baseline(spec, prompt):
    """One whole dense pass of the oracle on host cores, unsampled, in fp32 (the oracle's
    dtype parameter; numpy BLAS on every host thread): embedding, all layers at L = 512 and
    the LM head on the 32 rows of the active block.  Weight generation (the seeded input) is
    not timed; every step of the pass is."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import seeded_inputs as si
    from oracle import forward as of

    f32 = np.float32
    w = si.HostWeights(spec, 0, cache_layers=False)
    tokens = np.concatenate([prompt, np.full((1, G), spec.mask_id, np.int32)], axis=1)[0]
    L = tokens.shape[0]
    e = w.embed_rows(tokens)                           # input generation: not timed
    t0 = time.perf_counter()
    cos, sin = of.rope_tables(L, spec.head_dim, spec.rope_theta, f32)
    h = np.asarray(e, dtype=f32)
    t_pass = time.perf_counter() - t0
    for i in range(spec.n_layers):
        lw = w.layer(i)                                # input generation: not timed
        t0 = time.perf_counter()
        h = of.layer_forward(h, lw, spec, cos, sin, f32)
        t_pass += time.perf_counter() - t0
        del lw
        if i % 8 == 7:
            note(f"cpu baseline: {i + 1} of {spec.n_layers} layers")
    w.lm_head()                                        # input generation: not timed
    t0 = time.perf_counter()
    of.logits_from_hidden(w, spec, h[P:P + BLK], f32)
    t_pass += time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": round(1.0 / t_pass, 5), "unit": "passes/s", "cores": int(threads),
            "kind": "oracle", "nproc": os.cpu_count(),
            "sample": f"one whole fp32 oracle pass at L={L}, unsampled: embedding, all "
                      f"{spec.n_layers} layers, LM head on the {BLK} active-block rows; "
                      f"{t_pass:.2f} s per pass"}


def vocab_gate_roofline(iters=20):
    """HBM roofline of the vocab/gate kernel on bf16 logits [8, 512, 126464] (k = 1)."""
    import numpy as np
    import torch

    import seeded_inputs as si
    from paper_2608_11235_amd import DecodeState, Gate, Sched, vocab_gate
    w = si.vocab_gate_workload(seed=2)
    Bv, R, V = w.logits_bits.shape
    logits = torch.from_numpy(w.logits_bits.view(np.int16)).cuda()
    L = w.state["tokens"].shape[1]
    st = DecodeState.from_host(w.state, w.prompt_len, L - w.prompt_len, R, w.block_len)
    sc, gt = Sched(w.block_len, w.steps_per_block), Gate(DELTA_P, M_REQ, True)
    for _ in range(3):
        vocab_gate(logits, R, 0, V, w.mask_id, st, 1, sc, gt)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        vocab_gate(logits, R, 0, V, w.mask_id, st, 1, sc, gt)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    nbytes = Bv * R * V * 2
    ach = nbytes / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": counter_traffic("vocab_gate"),
            "us_per_launch": round(ms * 1e3, 2),
            "workload": "bf16 logits [8, 512, 126464], k = 1"}


def fidelity_run(m, prompt, gen_len, block_len, steps, delta_p, m_req, scope, dense=None):
    """Dense decode (gate off) and CORA decode (gate on, persistence scope `scope`) of the
    same prompts on model m, each timed by wall clock around cora_block_decode; then a
    step-by-step replay of the (deterministic) CORA decode that records every gate
    acceptance.  Returns executed passes, rho = CORA / dense passes, speedup, and the
    fidelity metrics against the dense endpoint: L^out, the fraction of generated
    positions whose final token differs (Eq. 12), and L^acc (Eq. 7): per prompt, the
    fraction of gate-accepted tokens that differ from the endpoint at their position (0 when
    the gate accepted nothing), averaged over the prompts.  `dense` reuses the output of an
    earlier dense decode of the same prompts (timed(...) below)."""
    import numpy as np
    import torch

    import seeded_inputs as si
    from paper_2608_11235_amd import DecodeState, Gate, Sched

    Bp, Pp = prompt.shape
    sched = Sched(block_len, steps)
    pr = torch.from_numpy(prompt).cuda()

    def timed(gate):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        y, passes, total = m.block_decode(pr, gen_len, sched, gate)
        dt = time.perf_counter() - t0
        return y.cpu().numpy(), passes, total, dt

    y_d, p_d, tot_d, dt_d = timed(Gate(delta_p, m_req, False)) if dense is None else dense
    gate = Gate(delta_p, m_req, True, scope)
    y, p, tot, dt = timed(gate)
    # replay, recording acceptances (decision 2) at the active block's positions
    st = DecodeState.from_host(si.initial_decode_state(prompt, gen_len, m.spec.mask_id), Pp,
                               gen_len, block_len if scope == 0 else gen_len, block_len)
    n_blocks = gen_len // block_len
    acc = [[] for _ in range(Bp)]
    while True:
        blk = st.block_idx.cpu().numpy().copy()
        if (blk >= n_blocks).all():
            break
        m.denoise_step(st, sched, gate)
        dec, tok = st.decision.cpu().numpy(), st.tokens.cpu().numpy()
        for b in range(Bp):
            if blk[b] < n_blocks:
                for j in np.nonzero(dec[b] == 2)[0]:
                    pos = Pp + int(blk[b]) * block_len + int(j)
                    acc[b].append((pos, int(tok[b, pos])))
    n_acc = sum(len(a) for a in acc)
    bad = [sum(int(t != y_d[b, i]) for i, t in acc[b]) for b in range(Bp)]
    l_acc = float(np.mean([bad[b] / len(acc[b]) if acc[b] else 0.0 for b in range(Bp)]))
    rho = float(p.sum()) / float(p_d.sum())
    return {
        "dense": {"passes": int(p_d.sum()), "wall_s": round(dt_d, 3),
                  "passes_per_s": round(tot_d / dt_d, 2)},
        "cora": {"passes": int(p.sum()), "passes_per_block": p.tolist(), "rho": round(rho, 4),
                 "inv_rho": round(1.0 / rho, 3), "wall_s": round(dt, 3),
                 "speedup_vs_dense": round(dt_d / dt, 3),
                 "L_out": float(np.mean(y[:, Pp:] != y_d[:, Pp:])), "accepted": n_acc,
                 "L_acc": l_acc,
                 "replay_matches_block_decode": bool((st.tokens.cpu().numpy() == y).all())},
        "arrays": {"dense_tokens": y_d, "cora_tokens": y, "dense_passes": p_d, "cora_passes": p,
                   "accepted": acc},
        "dense_run": (y_d, p_d, tot_d, dt_d),
    }


def gated_decode_leg(logit_scale=8.0):
    """Labelled gate-exercising run (not a paper configuration): the LLaDA-8B shape with
    random-init logits scaled x8, so top-1 confidences spread and the gate fires.  Dense vs
    CORA with the BLOCK and the GLOBAL persistence scope (fidelity_run).  With random
    weights a prediction depends on the whole committed context, so after the first
    acceptance the CORA trajectory leaves the dense one: L^out / L^acc measure that, not the
    fidelity a trained model would show."""
    from dataclasses import replace

    import seeded_inputs as si
    from paper_2608_11235_amd import LLADA_8B, Model

    spec = replace(LLADA_8B, logit_scale=logit_scale, name=f"llada8b-logits-x{logit_scale:g}")
    prompt = si.prompt_tokens(1, B, P, spec.vocab, spec.mask_id)
    out = {"label": f"LLaDA-8B shape, logits x{logit_scale:g} so the gate fires on random "
                    "weights; not a paper configuration", "gate": [DELTA_P, M_REQ]}
    with Model(spec, seed=0, max_batch=B, max_seq=P + G) as m:
        for name, scope in (("cora_block", 0), ("cora_global", 1)):
            r = fidelity_run(m, prompt, G, BLK, S, DELTA_P, M_REQ, scope)
            out["dense"] = r["dense"]
            c = r["cora"]
            c["L_out"], c["L_acc"] = round(c["L_out"], 4), round(c["L_acc"], 4)
            out[name] = c
    return out


def compaction_leg(batch=8, logit_scale=8.0):
    """Labelled batch-row compaction run (not a paper configuration): 8 prompts at the
    LLaDA-8B shape with logits x8, so rows accept tokens at different rates and finish at
    different passes.  The same gated block decode is timed with compaction on (finished
    rows leave the dense pass) and off (every row runs until the last one finishes).  At
    this shape the GEMM split-K and tile plans depend on the row count, so the two decodes
    round differently and, with random weights, part ways; tokens_equal reports that."""
    from dataclasses import replace

    import numpy as np
    import torch

    import seeded_inputs as si
    from paper_2608_11235_amd import LLADA_8B, Gate, Model, Sched

    spec = replace(LLADA_8B, logit_scale=logit_scale, name=f"llada8b-logits-x{logit_scale:g}")
    prompt = torch.from_numpy(si.prompt_tokens(3, batch, P, spec.vocab, spec.mask_id)).cuda()
    sched, gate = Sched(BLK, S), Gate(DELTA_P, M_REQ, True)
    out = {"label": f"LLaDA-8B shape, B={batch}, logits x{logit_scale:g} so the gate fires on "
                    "random weights; not a paper configuration", "gate": [DELTA_P, M_REQ]}
    with Model(spec, seed=0, max_batch=batch, max_seq=P + G) as m:
        m.block_decode(prompt, BLK, sched, gate)  # warm-up: one block
        res = {}
        for name, on in (("off", False), ("on", True)):
            m.set_compaction(on)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            y, passes, total = m.block_decode(prompt, G, sched, gate)
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            res[name] = (y.cpu().numpy(), passes, total, dt)
    rows = res["on"][1].sum(axis=1)
    out.update({
        "batch_passes": res["on"][2],
        "row_passes": [int(v) for v in rows],
        "row_passes_computed_on": int(rows.sum()),
        "row_passes_computed_off": int(res["off"][2] * batch),
        "decode_s_off": round(res["off"][3], 3), "decode_s_on": round(res["on"][3], 3),
        "speedup": round(res["off"][3] / res["on"][3], 3),
        "tokens_equal": bool((res["on"][0] == res["off"][0]).all()),
        "passes_equal": bool((res["on"][1] == res["off"][1]).all()),
    })
    return out


def shape_legs():
    """The two other workloads: LLaDA-8B long fixed-horizon run (prompt 256 + gen 1024, 1024
    steps, L = 1280) and Dream-7B at B = 8 (prompt 256 + gen 256, 256 steps)."""
    import seeded_inputs as si
    return {"llada8b_gen1024_decode": decode_leg("llada8b gen1024", si.LLADA_8B, 1, 256, 1024),
            "dream7b_b8_gen256_decode": decode_leg("dream7b b8", si.DREAM_7B, 8, 256, 256)}


def _timed_decode(m, pr, gen_len, sched, gate):
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    y, passes, total = m.block_decode(pr, gen_len, sched, gate)
    torch.cuda.synchronize()
    return y.cpu().numpy(), passes, total, time.perf_counter() - t0


def decode_leg(name, spec, b, p, g):
    """A whole gated block decode (gate (0.65, 1), BLOCK scope, batch-row compaction on) and
    the dense fixed-horizon decode (gate off) of the same seeded prompts, each timed by wall
    clock around cora_block_decode: executed passes (per block), the step ratio rho, time
    per executed pass and generated tokens/s.  Random-init weights put every top-1
    confidence near 1e-3, far below 0.65, so the gate accepts nothing and rho = 1 (reported
    as measured)."""
    import numpy as np
    import torch

    import seeded_inputs as si
    from paper_2608_11235_amd import Gate, Model, Sched

    prompt = torch.from_numpy(si.prompt_tokens(1, b, p, spec.vocab, spec.mask_id)).cuda()
    sched = Sched(BLK, S)
    runs = {}
    with Model(spec, seed=0, max_batch=b, max_seq=p + g) as m:
        m.block_decode(prompt, BLK, sched, Gate(DELTA_P, M_REQ, True))  # warm-up: one block
        for key, gate in (("cora", Gate(DELTA_P, M_REQ, True)),
                          ("dense", Gate(DELTA_P, M_REQ, False))):
            runs[key] = _timed_decode(m, prompt, g, sched, gate)
            note(f"{name}: {key} decode {runs[key][2]} passes in {runs[key][3]:.1f} s")
    fl = pass_flops(spec, b * (p + g), b * BLK, batch=b)
    out = {"batch": b, "prompt_len": p, "gen_len": g, "block_len": BLK, "steps_per_block": S,
           "total_steps": g // BLK * S, "gate": [DELTA_P, M_REQ], "pass_tflop": round(fl / 1e12, 4)}
    for key, (y, passes, total, dt) in runs.items():
        ms = dt / total * 1e3
        out[key] = {"passes": int(passes.sum()), "batch_passes": int(total),
                    "passes_per_block_row0": passes[0].tolist(), "wall_s": round(dt, 3),
                    "ms_per_pass": round(ms, 3), "passes_per_s": round(total / dt, 3),
                    "gen_tokens_per_s": round(b * g / dt, 3),
                    "pass_mfma_frac": round(fl / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
    out["rho"] = round(float(runs["cora"][1].sum()) / float(runs["dense"][1].sum()), 4)
    out["tokens_equal_dense"] = bool((runs["cora"][0] == runs["dense"][0]).all())
    out["note"] = ("random-init weights: top-1 confidence ~1e-3, so the gate never reaches "
                   "0.65 and rho = 1")
    torch.cuda.empty_cache()
    return out


def table3_sweep_leg(logit_scale=8.0):
    """Labelled gate-variant sweep (the Table 3 ablation's settings; not a paper
    configuration): the LLaDA-8B shape, batch 1, gen 256, logits x8 so the gate fires on
    random weights.  One dense decode, then CORA with confidence only (m = 0), the default
    (delta_p 0.65, m = 1), two checks (m = 2), persistence only (delta_p = 0, m = 1) and the
    thresholds delta_p 0.5 and 0.8 (m = 1): rho, wall-clock speedup against 1/rho, L^acc
    (Eq. 7, per-prompt mean) and L^out (Eq. 12)."""
    from dataclasses import replace

    import seeded_inputs as si
    from paper_2608_11235_amd import LLADA_8B, Model

    spec = replace(LLADA_8B, logit_scale=logit_scale, name=f"llada8b-logits-x{logit_scale:g}")
    prompt = si.prompt_tokens(1, B, P, spec.vocab, spec.mask_id)
    variants = (("m0", 0.65, 0), ("m1", 0.65, 1), ("m2", 0.65, 2), ("persistence_only", 0.0, 1),
                ("dp0.5_m1", 0.5, 1), ("dp0.8_m1", 0.8, 1))
    out = {"label": f"LLaDA-8B shape, B=1, gen 256, logits x{logit_scale:g} so the gate fires on "
                    "random weights; the settings of the gate ablation, not a paper "
                    "configuration", "scope": "block"}
    dense = None
    with Model(spec, seed=0, max_batch=B, max_seq=P + G) as m:
        for name, dp, mr in variants:
            r = fidelity_run(m, prompt, G, BLK, S, dp, mr, 0, dense=dense)
            dense = r["dense_run"]
            out["dense"] = r["dense"]
            c = r["cora"]
            out[name] = {"delta_p": dp, "m_req": mr, "passes": c["passes"], "rho": c["rho"],
                         "speedup_vs_dense": c["speedup_vs_dense"],
                         "speedup_over_inv_rho": round(c["speedup_vs_dense"] * c["rho"], 4),
                         "L_acc": round(c["L_acc"], 4), "L_out": round(c["L_out"], 4),
                         "accepted": c["accepted"]}
            note(f"table-3 sweep: {name} rho {c['rho']}")
    return out


def shape_passes_leg(passes=6, warmup=2):
    """Per-pass wall-clock timing of whole denoising steps at the Dream-7B B = 8 and LLaDA-8B
    L = 1280 shapes (a short run for kernel traces of those shapes; the decode legs time the
    full decodes)."""
    import torch

    import seeded_inputs as si
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched

    out = {}
    for name, spec, b, p, g in (("dream7b_b8_gen256", si.DREAM_7B, 8, 256, 256),
                                ("llada8b_gen1024", si.LLADA_8B, 1, 256, 1024)):
        prompt = si.prompt_tokens(1, b, p, spec.vocab, spec.mask_id)
        sched, gate = Sched(BLK, S), Gate(DELTA_P, M_REQ, True)
        with Model(spec, seed=0, max_batch=b, max_seq=p + g) as m:
            st = DecodeState.from_host(si.initial_decode_state(prompt, g, spec.mask_id), p, g,
                                       BLK, BLK, device="cuda")
            for _ in range(warmup):
                m.denoise_step(st, sched, gate)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(passes):
                m.denoise_step(st, sched, gate)
            torch.cuda.synchronize()
            dt = (time.perf_counter() - t0) / passes
        fl = pass_flops(spec, b * (p + g), b * BLK, batch=b)
        out[name] = {"passes_timed": passes, "ms_per_pass": round(dt * 1e3, 3),
                     "pass_mfma_frac": round(fl / dt / 1e12 / PEAK_BF16_TFLOPS, 4)}
        torch.cuda.empty_cache()
        note(f"shape passes {name} done")
    return out


def copy_calibration(nbytes=1 << 30, iters=5):
    """A plain device-to-device copy of known size: reference for HBM byte counters."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "iters": iters,
                      "us_per_copy": round(ms * 1e3, 2),
                      "GB_per_s_read_plus_write": round(2 * nbytes / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-vocab", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-gated", action="store_true",
                    help="skip the labelled logits-x8 gated-decode leg")
    ap.add_argument("--no-compaction", action="store_true",
                    help="skip the labelled B=8 batch-row compaction leg")
    ap.add_argument("--no-shapes", action="store_true",
                    help="skip the gated vs dense decodes at the LLaDA-8B gen-1024 and "
                         "Dream-7B B=8 workloads")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the labelled logits-x8 gate-variant sweep")
    ap.add_argument("--only", choices=["all", "pass", "vocab", "copy", "gated", "compaction",
                                       "shapes", "shape-passes", "sweep", "cpu"],
                    default="all",
                    help="run one leg only (profiling runs): the timed passes, the vocab/gate "
                         "kernel, or a plain 1 GiB device copy that calibrates byte counters")
    args = ap.parse_args()
    if args.only == "copy":
        copy_calibration()
        return
    if args.only == "vocab":
        print(json.dumps({"vocab_gate_roofline": vocab_gate_roofline()}), flush=True)
        return
    if args.only == "gated":
        print(json.dumps({"gated_decode_logits_x8": gated_decode_leg()}), flush=True)
        return
    if args.only == "compaction":
        print(json.dumps({"compaction_b8_logits_x8": compaction_leg()}), flush=True)
        return
    if args.only == "shapes":
        print(json.dumps(shape_legs()), flush=True)
        return
    if args.only == "shape-passes":
        print(json.dumps({"shape_passes": shape_passes_leg()}), flush=True)
        return
    if args.only == "sweep":
        print(json.dumps({"table3_sweep_logits_x8": table3_sweep_leg()}), flush=True)
        return
    if args.only == "cpu":
        import seeded_inputs as si_
        prompt = si_.prompt_tokens(1, B, P, si_.LLADA_8B.vocab, si_.LLADA_8B.mask_id)
        print(json.dumps({"cpu_baseline": cpu_baseline(si_.LLADA_8B, prompt)}), flush=True)
        return
    if args.only == "pass":
        args.no_decode = args.no_vocab = args.no_cpu_baseline = args.no_gated = True
        args.no_compaction = args.no_shapes = args.no_sweep = True
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (batch rows "
              "decode independently, so more GPUs shard rows with no collective)", file=sys.stderr)
        sys.exit(2)
    if args.warmup + args.steps > G:
        sys.exit("warmup + steps must fit in one 256-pass decode")

    import numpy as np
    import torch

    import seeded_inputs as si
    from paper_2608_11235_amd import LLADA_8B, DecodeState, Gate, Model, Sched

    spec = LLADA_8B
    dev = torch.device("cuda:0")
    prompt = si.prompt_tokens(1, B, P, spec.vocab, spec.mask_id)
    t_create = time.perf_counter()
    model = Model(spec, seed=0, max_batch=B, max_seq=P + G)
    t_create = time.perf_counter() - t_create
    sched, gate = Sched(BLK, S), Gate(DELTA_P, M_REQ, True)
    host = si.initial_decode_state(prompt, G, spec.mask_id)
    st = DecodeState.from_host(host, P, G, BLK, BLK, device=dev)

    for _ in range(args.warmup):
        model.denoise_step(st, sched, gate)
    torch.cuda.synchronize()
    unres0 = int(st.unresolved.sum())
    model.read_timing()  # clear
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        # the gate/up launches of every TIME_EVERY-th timed pass are stamped with HIP events
        # (each stamp adds a few us of dispatch gap, so stamping every pass would tax the
        # pass rate being measured)
        model.set_timing(i % TIME_EVERY == 0)
        model.denoise_step(st, sched, gate)
    model.set_timing(False)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    gu_ms, gu_launches = model.read_timing()
    note(f"timed passes done: {args.steps} in {t1 - t0:.3f} s")
    elapsed = t1 - t0
    committed = unres0 - int(st.unresolved.sum())
    passes_per_s = args.steps / elapsed
    ms_per_step = elapsed * 1e3 / args.steps
    M = B * (P + G)
    fl_pass = pass_flops(spec, M, B * BLK)
    gu_avg_ms = gu_ms / max(1, gu_launches)
    gu_tflops = gu_flops(spec, M) / (gu_avg_ms * 1e-3) / 1e12

    result = {
        "metric": "denoising passes/s + gen tokens/s, LLaDA-8B shape gen256; MFMA util %",
        "value": round(passes_per_s, 3),
        "unit": "passes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random prompts, seeded N(0,0.02) weights)",
        "config": {"workload": "llada8b-gen256", "batch": B, "prompt_len": P, "gen_len": G,
                   "block_len": BLK, "steps_per_block": S, "gate": [DELTA_P, M_REQ]},
        "gen_tokens_per_s": round(committed / elapsed, 3),
        "pass_tflop": round(fl_pass / 1e12, 4),
        "pass_mfma_frac": round(fl_pass / (ms_per_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "roofline": {"bound": "mfma", "achieved": round(gu_tflops, 1), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gu_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": counter_traffic("gate_up"),
                     "kernel": "gate/up SwiGLU GEMM (M 512, N 24576, K 4096)",
                     "us_per_launch": round(gu_avg_ms * 1e3, 2), "launches": gu_launches},
        "model_create_s": round(t_create, 2),
    }

    if not args.no_decode:
        pr = torch.from_numpy(prompt).to(dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        out, passes, total = model.block_decode(pr, G, sched, gate)
        dt = time.perf_counter() - t0
        dense = np.full_like(passes, S)
        result["block_decode"] = {
            "wall_s": round(dt, 3), "passes": int(passes.sum()), "dense_passes": int(dense.sum()),
            "rho": round(float(passes.sum() / dense.sum()), 4),
            "passes_per_s": round(int(total) / dt, 3), "gen_tokens_per_s": round(B * G / dt, 3),
            "note": "random-init weights: top-1 confidence ~1e-3, so the gate never reaches 0.65",
        }
    model.close()
    del model
    torch.cuda.empty_cache()

    if not args.no_decode:
        note("block decode leg done")
    if not args.no_vocab:
        result["vocab_gate_roofline"] = vocab_gate_roofline()
        note("vocab/gate leg done")
    if not args.no_gated:
        result["gated_decode_logits_x8"] = gated_decode_leg()
        note("gated decode leg done")
    if not args.no_compaction:
        result["compaction_b8_logits_x8"] = compaction_leg()
        note("compaction leg done")
    if not args.no_sweep:
        result["table3_sweep_logits_x8"] = table3_sweep_leg()
        note("gate-variant sweep leg done")
    if not args.no_shapes:
        result.update(shape_legs())
    if not args.no_cpu_baseline:
        note("cpu baseline leg starts")
        import seeded_inputs as si_
        try:
            result["cpu_baseline"] = cpu_baseline(si_.LLADA_8B, prompt)
        except Exception as e:  # report, do not lose the GPU line
            result["cpu_baseline"] = {"error": repr(e)}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
