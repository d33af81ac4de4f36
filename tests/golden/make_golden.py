"""Writes the golden oracle scores under tests/golden/ (calls only oracle/).

The paper prints no worked numeric example, so these files are regression pins
of the fp64 oracle on the tiny fp32 workload (1 request, L=256, S=8, C=16,
d=64, 2 heads, 1 encoder + 1 decoder layer), for the base weights and for the
"sharp"+"affine" weight variant. Run from the repository root:
    python tests/golden/make_golden.py
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_2607_28940_amd import inputs as I  # noqa: E402


def main():
    O.build()
    wl = I.workload("tiny")
    here = os.path.dirname(os.path.abspath(__file__))
    for variant, fn in (((), "tiny_scores.txt"), (("sharp", "affine"), "tiny_sharp_affine_scores.txt")):
        w = I.make_weights(wl.model, variant)
        Xb = I.request_tokens(wl, 0, I.STREAM_BEHAVIOR)
        Xs = I.request_tokens(wl, 0, I.STREAM_SERVING)
        Xc = I.request_tokens(wl, 0, I.STREAM_CANDIDATES)
        s, _ = O.Oracle(wl.model, w).run_request(Xb, Xs, Xc)
        hdr = ("TransX oracle candidate logits, tiny fp32 workload, weights variant %s; "
               "Sec. 4.1 model, linear scalar head (k=2 case of Eq. action-decoding)" % (list(variant) or "base"))
        np.savetxt(os.path.join(here, fn), s, fmt="%.17e", header=hdr)


if __name__ == "__main__":
    main()
