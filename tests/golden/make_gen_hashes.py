"""Write tests/golden/gen_sha256.json: SHA-256 of every generated array.

Run from the repository root: python tests/golden/make_gen_hashes.py
It calls only the seeded input generator (``workloads``); the stored digests
guard the draw order and rounding of the synthetic inputs against drift.
"""
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from workloads import make_attn_batch, make_decode_inputs  # noqa: E402

FIELDS = ("prefix_len", "branch_page", "num_new", "past_len", "q", "shared_k", "shared_v", "priv_k", "priv_v")


def digest(a):
    a = np.ascontiguousarray(a)
    return hashlib.sha256(a.tobytes() + str(a.dtype).encode() + str(a.shape).encode()).hexdigest()


def attn_digests(name, seed):
    b = make_attn_batch(name, seed)
    return {f: digest(getattr(b, f)) for f in FIELDS}


def decode_digests(seed, layers=1):
    d = make_decode_inputs("c4", seed, num_layers=layers)
    out = {f: digest(getattr(d, f)) for f in ("prefix_len", "branch_page", "num_new", "past_len", "hidden_in")}
    for f in ("shared_k", "shared_v", "priv_k", "priv_v", "w_qkv", "w_o", "w_gate", "w_up", "w_down"):
        out[f] = [digest(x) for x in getattr(d, f)]
    return out


def all_digests():
    res = {}
    for name in ("c1", "c2", "c3", "c5"):
        for seed in (0, 1, 2):
            res[f"{name}/seed{seed}"] = attn_digests(name, seed)
    res["c4_1layer/seed0"] = decode_digests(0)
    return res


if __name__ == "__main__":
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "gen_sha256.json")
    with open(path, "w") as f:
        json.dump(all_digests(), f, indent=1, sort_keys=True)
    print("wrote", path)
