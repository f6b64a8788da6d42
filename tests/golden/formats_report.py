"""Writes formats_report.txt: for every tensor of the synthetic workloads, the
Eq. 3 bias and the FP8 codes in the paper's formats (Table 7 rows "(a)") and in
the OCP formats the matrix cores consume (rows "(b)"), each with its own AMAX
bias, and how many elements are represented differently.  Calls only the
oracle.  Tensors above 2^24 elements are reported on their first rows (stated
per line).  Run from the repository root:
    python tests/golden/formats_report.py
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import oracle  # noqa: E402
from paper_2309_17224_amd import workloads as wl  # noqa: E402

CAP = 1 << 24


def bits(t):
    return t.contiguous().view(__import__("torch").int16).numpy().view(np.uint16)


def main():
    lines = ["# FP8 formats (a) vs (b) on the synthetic workloads (oracle)", "",
             "Each tensor is cast with its own AMAX bias in the paper's format (a) and in the OCP format (b).",
             "E4: the biases differ by one unless the amax mantissa lies in (1.75, 1.875]; with that offset the",
             "codes are the same except -0 (0x80 in (b), 0x00 in (a)) and no represented value changes; with",
             "equal biases the codes move by one binade and the values that differ are (b) subnormals.",
             "E5: the biases are always equal, every code moves by one binade, and only values below the",
             "smallest (b) normal can be represented differently (none in these tensors).", "",
             "tensor: shape [rows used] | fmt | bias (b) | bias (a) | codes differing | represented values differing", ""]
    for w in wl.WORKLOADS.values():
        for t in w.tensors:
            x = wl.make_tensor(w, t.name)
            rows = x.shape[0] if x.numel() <= CAP else max(1, CAP // x.shape[1])
            xb = bits(x[:rows])
            # the method's format for the tensor: E5 for gradients, E4 otherwise (App. B)
            kinds = [("E5", 1, 3)] if t.name.lower().startswith("dy") else [("E4", 0, 2)]
            for name, fb, fa in kinds:
                bb, _, _ = oracle.scale_bias(xb, fb)
                ba, _, _ = oracle.scale_bias(xb, fa)
                qb, qa = oracle.cast(xb, fb, bb), oracle.cast(xb, fa, ba)
                vb = oracle.decode_table(fb)[qb].astype(np.float64) * 2.0 ** -bb
                va = oracle.decode_table(fa)[qa].astype(np.float64) * 2.0 ** -ba
                n = qb.size
                lines.append(f"{w.name}/{t.name}: {tuple(x.shape)} [{rows}] | {name} | {bb} | {ba} | "
                             f"{np.count_nonzero(qa != qb) / n:.3%} | {np.count_nonzero(va != vb) / n:.3%}")
    out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "formats_report.txt")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
