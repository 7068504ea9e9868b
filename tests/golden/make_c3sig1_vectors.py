"""Writes c3sig1_vectors.txt, the known-answer vectors of C3SIG-1.

Run from the repository root: ``python tests/golden/make_c3sig1_vectors.py``.
Every value comes from the oracle (``oracle/``) alone; the chunk bytes come
from ``workloads.lcg_bytes`` (a 32-bit LCG pattern), so the file needs only
the seed to rebuild them.  Any change to these values is a change of the
signature's definition and must re-freeze the file deliberately.
"""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle      # noqa: E402
import workloads   # noqa: E402

F32, BF16, F16, RAW = oracle.F32, oracle.BF16, oracle.F16, oracle.RAW
NAMES = {F32: "F32", BF16: "BF16", F16: "F16", RAW: "RAW"}

# (name, dtype, shape, chunk_bytes, seed): every chunk of each tensor gets a
# chunk line, and each tensor a tensor line.
TENSORS = [
    ("raw_empty", RAW, (0,), 1024, 1),
    ("f32_zero_dim", F32, (4, 0), 1024, 2),
    ("raw_1", RAW, (1,), 1024, 3),
    ("raw_15", RAW, (15,), 1024, 4),
    ("raw_16", RAW, (16,), 1024, 5),
    ("raw_17", RAW, (17,), 1024, 6),
    ("bf16_scalar", BF16, (), 1024, 7),
    ("f32_3x5", F32, (3, 5), 1024, 8),
    ("f16_2x3x7", F16, (2, 3, 7), 1024, 9),
    ("f32_one_key_period", F32, (256,), 1024, 10),
    ("f32_four_blocks", F32, (1000,), 4096, 11),
    ("f32_three_chunks", F32, (3000,), 4096, 12),
    ("bf16_64x100", BF16, (64, 100), 2048, 13),
    ("raw_two_chunks", RAW, (10000,), 8192, 14),
    ("f32_multi_tile", F32, (8192,), 32768, 15),
    ("f16_4d", F16, (2, 2, 2, 1024), 4096, 16),
    ("raw_8d", RAW, (1, 2, 1, 2, 1, 2, 1, 2), 1024, 17),
    ("bf16_ragged_odd", BF16, (3, 1111), 2048, 18),
]


def shape_text(shape):
    return ",".join(str(d) for d in shape) if shape else "scalar"


def main():
    lines = [
        "# Known-answer vectors of C3SIG-1 (Sec. 5.2 asks for a deterministic,",
        "# position-sensitive 64-bit hash over dtype, shape and bytes; C3SIG-1 is this",
        "# implementation's construction).  Written by make_c3sig1_vectors.py from the",
        "# oracle.  Tensor bytes: workloads.lcg_bytes(seed, nbytes).",
        "# chunk  | name | dtype | shape | chunk_bytes | seed | k | n | A | B | sig",
        "# tensor | name | dtype | shape | chunk_bytes | seed | chunks | tensor_sig",
    ]
    for name, dt, shape, cb, seed in TENSORS:
        nb = oracle.ELEM_SIZE[dt]
        for d in shape:
            nb *= d
        data = workloads.lcg_bytes(seed, nb)
        meta = [(dt, shape)]
        rec = oracle.signature([[data]], meta, cb)
        C = rec["sig"].shape[1]
        for k in range(C):
            chunk = data[k * cb:min(nb, (k + 1) * cb)]
            A, B = oracle.nh(chunk)
            sig = int(rec["sig"][0, k])
            lines.append(f"chunk | {name} | {NAMES[dt]} | {shape_text(shape)} | {cb} | {seed} | "
                         f"{k} | {chunk.size} | {A:016x} | {B:016x} | {sig:016x}")
        tsig = int(oracle.tensor_signature(rec, 1)[0, 0])
        lines.append(f"tensor | {name} | {NAMES[dt]} | {shape_text(shape)} | {cb} | {seed} | "
                     f"{C} | {tsig:016x}")
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c3sig1_vectors.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(path)


if __name__ == "__main__":
    main()
