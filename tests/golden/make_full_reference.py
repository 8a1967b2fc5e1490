"""Write the float64 oracle's free-running greedy run of a full-size workload
configuration to tests/golden/full/<config>.npz.

    python tests/golden/make_full_reference.py 8b_long [32b ...]

Only `oracle/` computes here.  The seeded input generator (`inputs`, which does
no arithmetic of the forward pass) and the configuration table supply the
weights and the prompt, exactly as the GPU test receives them.  For 8-bit
configurations the weights are quantised with the oracle's own rule
(`oracle.quantize_q8`).  Their exact values q*d (at most 19 significant bits)
are then held as float32.

The oracle prefills the prompt in the configuration's chunks.  It then runs the
configuration's decode steps, each feeding back its own argmax (a free-running
greedy run; nothing from the GPU path goes in).  Per generated step s
(0 = the prefill's token) the file keeps:
- ids[s]                         the oracle's greedy id (lowest index on ties)
- max_abs[s]                     max_i |o_i|: the scale of the logit tolerance
- top_idx[s, :8], top_val[s, :8] the eight largest logits, in decreasing order
                                 (ties broken by lower index)
- sample_val[s, :]               the logits at 128 fixed indices ``sample_idx``,
                                 drawn without replacement from
                                 default_rng([7, config key])
- full_logits                    the whole logit vector (stored as float32) at
                                 the steps in ``full_steps``: the prefill and
                                 the last step
plus ``meta`` (JSON): the configuration, the seeds, digests of the prompt, of
sampled weight values and of the oracle sources.  The test checks the prompt
and weight digests before it compares anything.

The script prints one line per prefill layer and per decode step.
"""

from __future__ import annotations

import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import DecoderOracle, dequantize_q8, greedy, quantize_q8  # noqa: E402
from oracle.native import StoredWeights  # noqa: E402
from paper_2608_24204_amd import configs, inputs  # noqa: E402

OUT_DIR = os.path.join(ROOT, "tests", "golden", "full")
TOPK = 8
N_SAMPLE = 128
SAMPLE_SEED = 7
ORACLE_SOURCES = ["oracle/model.py", "oracle/native.py", "oracle/matvec.c", "oracle/quant.py"]


def sample_indices(cfg) -> np.ndarray:
    rng = np.random.default_rng([SAMPLE_SEED, cfg.key])
    return np.sort(rng.choice(cfg.vocab, N_SAMPLE, replace=False)).astype(np.int32)


def prompt_digest(prompt) -> str:
    return hashlib.sha256(np.asarray(prompt, np.int32).tobytes()).hexdigest()


def weight_digest(weights) -> str:
    """sha256 over the first and last 4096 stored values of every matrix, in
    name order (catches a change of the generator, its seeds or its layout)."""
    h = hashlib.sha256()
    for name in sorted(weights):
        a = np.asarray(weights[name])
        if a.ndim != 2:
            continue
        flat = a.reshape(-1)
        h.update(name.encode())
        h.update(np.ascontiguousarray(flat[:4096]).tobytes())
        h.update(np.ascontiguousarray(flat[-4096:]).tobytes())
    return h.hexdigest()


def oracle_digest() -> str:
    h = hashlib.sha256()
    for rel in ORACLE_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def top_k(o: np.ndarray, k: int):
    """Indices of the k largest values, decreasing, lower index first on ties."""
    idx = np.lexsort((np.arange(o.size), -o))[:k]
    return idx.astype(np.int32), o[idx]


def quantised_store(weights, threads: int) -> dict:
    """Matrices replaced by their exact 8-bit values q*d as float32 (the oracle's
    own quantisation); each source tensor is dropped once converted."""
    names = [n for n, a in weights.items() if np.asarray(a).ndim == 2]

    def one(name):
        src = inputs.bf16_bits_to_f32(weights[name]) if weights[name].dtype == np.uint16 \
            else weights[name].astype(np.float32)
        q, d = quantize_q8(src)
        del src
        return name, dequantize_q8(q, d).astype(np.float32)

    out = {n: a for n, a in weights.items() if np.asarray(a).ndim != 2}
    with ThreadPoolExecutor(threads) as ex:
        for name, a in ex.map(one, names):
            out[name] = a
            weights[name] = None
    return out


def run(name: str, out_dir: str = OUT_DIR) -> str:
    cfg = configs.CONFIGS[name]
    t0 = time.time()
    threads = min(16, os.cpu_count() or 1)
    w = inputs.make_weights(cfg, threads=threads)
    prompt = inputs.make_prompt(cfg)
    wdig = weight_digest(w)
    print(f"[{name}] weights generated ({time.time() - t0:.0f} s)", flush=True)
    if cfg.weight_dtype == "q8":
        w = quantised_store(w, threads)
        print(f"[{name}] quantised ({time.time() - t0:.0f} s)", flush=True)
    orc = DecoderOracle(cfg, StoredWeights(w), max_seq=cfg.max_seq)

    n_steps = cfg.decode_steps
    V = cfg.vocab
    sidx = sample_indices(cfg)
    ids = np.zeros(n_steps + 1, np.int32)
    max_abs = np.zeros(n_steps + 1)
    top_idx = np.zeros((n_steps + 1, TOPK), np.int32)
    top_val = np.zeros((n_steps + 1, TOPK))
    sample_val = np.zeros((n_steps + 1, N_SAMPLE))
    full_steps = np.array([0, n_steps], np.int32)
    full = np.zeros((2, V), np.float32)

    def record(s, o):
        ids[s] = greedy(o)
        max_abs[s] = np.max(np.abs(o))
        top_idx[s], top_val[s] = top_k(o, TOPK)
        sample_val[s] = o[sidx]
        for j, fs in enumerate(full_steps):
            if s == fs:
                full[j] = o.astype(np.float32)

    t1 = time.time()
    chunk = cfg.prefill_chunk
    o = None
    for c0 in range(0, len(prompt), chunk):
        part = prompt[c0:c0 + chunk]
        o = orc.forward(part, progress=lambda l, c0=c0: print(
            f"[{name}] prefill rows {c0}..{c0 + len(part) - 1}: layer {l + 1}/{cfg.n_layers} "
            f"({time.time() - t1:.0f} s)", flush=True))
    record(0, o)
    t2 = time.time()
    for s in range(1, n_steps + 1):
        o = orc.forward([int(ids[s - 1])])
        record(s, o)
        if s % 8 == 0 or s == n_steps:
            print(f"[{name}] decode step {s}/{n_steps} ({time.time() - t2:.0f} s)", flush=True)
    meta = {"config": name, "prompt_len": cfg.prompt_len, "decode_steps": n_steps, "vocab": V,
            "weight_seed": inputs.WEIGHT_SEED, "prompt_seed": inputs.PROMPT_SEED,
            "prefill_chunk": chunk, "kv_round": orc.kv_round,
            "prompt_sha256": prompt_digest(prompt), "weights_sha256": wdig,
            "oracle_sha256": oracle_digest(), "topk": TOPK, "sample_seed": SAMPLE_SEED,
            "prefill_s": round(t2 - t1, 1), "decode_s": round(time.time() - t2, 1)}
    os.makedirs(out_dir, exist_ok=True)
    path = os.path.join(out_dir, f"{name}.npz")
    tmp = path + ".tmp.npz"
    np.savez_compressed(tmp, meta=np.array(json.dumps(meta)), ids=ids, max_abs=max_abs,
                        top_idx=top_idx, top_val=top_val, sample_idx=sidx,
                        sample_val=sample_val, full_steps=full_steps, full_logits=full)
    os.replace(tmp, path)
    margins = top_val[:, 0] - top_val[:, 1]
    print(f"[{name}] wrote {path}: {n_steps + 1} ids, min oracle margin "
          f"{margins.min():.3g} at step {int(margins.argmin())}, total "
          f"{time.time() - t0:.0f} s", flush=True)
    return path


if __name__ == "__main__":
    args = sys.argv[1:]
    out = OUT_DIR
    if "--out" in args:
        i = args.index("--out")
        out = args[i + 1]
        del args[i:i + 2]
    if not args:
        sys.exit(__doc__)
    for n in args:
        run(n, out)
