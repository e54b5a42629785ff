"""Writes the golden stream fixtures from the CPU oracle (and nothing else).

Run from the repository root: ``python tests/golden/make_golden.py``.
Each fixture is a small seeded input and the stream the oracle produces for
it; the test suite re-creates both and checks the bytes, so that any later
change to the oracle's arithmetic shows up as a fixture diff that has to be
justified.
"""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import ref  # noqa: E402
import workloads as W  # noqa: E402

# (name, input, dtype, block bytes, table mode)
CASES = [
    ("normal_bf16_5000_b4096", lambda: W.normal_bf16(5000, seed=7), "bf16", 4096, "per_block"),
    ("grad_fp32_3000_b4096", lambda: W.grad_fp32(3000, seed=7), "fp32", 4096, "per_block"),
    ("grad_fp16_6000_b4096", lambda: W.grad_fp16(6000, seed=7), "fp16", 4096, "per_block"),
    ("normal_e4m3fn_6000_b4096", lambda: W.normal_fp8_pairs(6000, "e4m3fn", seed=7), "e4m3fn", 4096, "per_block"),
    ("normal_e5m2_6000_b4096", lambda: W.normal_fp8_pairs(6000, "e5m2", seed=7), "e5m2", 4096, "per_block"),
    ("normal_bf16_5000_b4096_sampled", lambda: W.normal_bf16(5000, seed=7), "bf16", 4096, "sampled"),
]


def main():
    out = {}
    for name, gen, dtype, bb, mode in CASES:
        x = gen()
        s = ref.compress_table(x, dtype, bb, mode)
        out[name] = dict(dtype=dtype, block_bytes=bb, n=int(x.size), table_mode=mode,
                         input_sha256=hashlib.sha256(x.tobytes()).hexdigest(),
                         stream_bytes=int(s.size),
                         stream_sha256=hashlib.sha256(s.tobytes()).hexdigest())
        with open(os.path.join(HERE, name + ".hex"), "w") as fh:
            h = s.tobytes().hex()
            fh.write("\n".join(h[i:i + 64] for i in range(0, len(h), 64)) + "\n")
    with open(os.path.join(HERE, "streams.json"), "w") as fh:
        json.dump(out, fh, indent=1, sort_keys=True)


if __name__ == "__main__":
    main()
