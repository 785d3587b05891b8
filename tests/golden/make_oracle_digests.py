"""Write tests/golden/oracle_digests.json: SHA-256 digests of the oracle's full
outputs on the large model-shaped workloads, where recomputing every output
inside a GPU test would take minutes of CPU time.

Only the oracle (``oracle/``) and the seeded input generators
(``paper_2502_19405_amd/inputs.py``) run here; nothing from the GPU library is
imported.  Each workload's entry records the SHA-256 of every input, of the
oracle sources that produced it, and of every output (float32, row-major,
little-endian bytes).  The GPU tests hash their own outputs and compare.

    python tests/golden/make_oracle_digests.py [workload ...]

Workloads: llama_attention (4 x 1024 tokens, d 4096, 32 heads: Q, K, V, scores
-- whole and with +0 above each head's diagonal --, probabilities, head outputs,
output projection), llama_linear_backward (8192
tokens, 4096 -> 14336: dX and dW), mlp_train_step_4096 (two training steps of
the DistilBERT feed-forward block at 4096 tokens).
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from oracle import compose  # noqa: E402
from paper_2502_19405_amd import inputs  # noqa: E402

OUT = os.path.join(HERE, "oracle_digests.json")
ORACLE_SOURCES = ("repops_ref.c", "compose.py", "__init__.py")


def sha256_of(a) -> str:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return hashlib.sha256(a.astype("<f4", copy=False).tobytes()).hexdigest()


def oracle_source_sha256() -> str:
    h = hashlib.sha256()
    for f in ORACLE_SOURCES:
        with open(os.path.join(ROOT, "oracle", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def train_step_gradients(tokens, step_count=2):
    """The loss gradients of the training-step workload: drawn after the
    block's inputs from their own seeded stream, one [tokens, 768] array per
    step, N(0, 1e-4)."""
    g = inputs.rng(1100 + tokens)
    return [inputs.normal(g, (tokens, 768), var=1e-4) for _ in range(step_count)]


def causal_lower(S):
    """The scores at or below each head's diagonal, +0 above it (the part a
    causal softmax reads)."""
    T = S.shape[-1]
    return np.where(np.tril(np.ones((T, T), bool)), S, np.float32(0.0)).astype(np.float32)


def llama_attention():
    d = inputs.llama_attention()
    out = compose.attention_forward(d["X"], d["Wq"], d["Wk"], d["Wv"], d["Wo"], 4, 1024, 32)
    digests = {k: sha256_of(v) for k, v in out.items()}
    digests["S_lower"] = sha256_of(causal_lower(out["S"]))
    return d, digests


def llama_linear_backward():
    d = inputs.llama_linear_backward()
    dX, dW = compose.linear_backward(d["X"], d["dY"], d["W"])
    return d, {"dX": sha256_of(dX), "dW": sha256_of(dW)}


def mlp_train_step_4096():
    tokens = 4096
    d = inputs.distilbert_mlp(tokens=tokens)
    P = [d[k] for k in compose.MLP_PARAM_NAMES]
    n = sum(p.size for p in P)
    M, V = np.zeros(n, np.float32), np.zeros(n, np.float32)
    dYs = train_step_gradients(tokens)
    outs = {}
    for step, dY in enumerate(dYs, start=1):
        Y, dX, grads, P, M, V = compose.mlp_train_step(P, M, V, d["X"], dY, step)
        outs[f"step{step}/Y"] = sha256_of(Y)
        outs[f"step{step}/dX"] = sha256_of(dX)
        for name, gr, p in zip(compose.MLP_PARAM_NAMES, grads, P):
            outs[f"step{step}/grad_{name}"] = sha256_of(gr)
            outs[f"step{step}/param_{name}"] = sha256_of(p)
        outs[f"step{step}/exp_avg"] = sha256_of(M)
        outs[f"step{step}/exp_avg_sq"] = sha256_of(V)
    ins = dict(d)
    for i, dY in enumerate(dYs, start=1):
        ins[f"dY_step{i}"] = dY
    return ins, outs


WORKLOADS = {
    "llama_attention": llama_attention,
    "llama_linear_backward": llama_linear_backward,
    "mlp_train_step_4096": mlp_train_step_4096,
}


def main(names):
    assert oracle.env_check() == 0, "host floating-point environment is not strict IEEE"
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as fh:
            data = json.load(fh)
    for name in names or list(WORKLOADS):
        t0 = time.perf_counter()
        ins, outs = WORKLOADS[name]()
        data[name] = {
            "oracle_sources_sha256": oracle_source_sha256(),
            "inputs_sha256": {k: sha256_of(v) for k, v in ins.items()},
            "outputs_sha256": outs,
        }
        print(f"{name}: {len(outs)} outputs in {time.perf_counter() - t0:.0f} s", flush=True)
        with open(OUT, "w") as fh:
            json.dump(data, fh, indent=1, sort_keys=True)
            fh.write("\n")


if __name__ == "__main__":
    main(sys.argv[1:])
