"""Writes the oracle's segmentation of the 8B-shaped 8K and 32K workloads
(seed 0) to segment_<config>.txt: the slot starts of the DP (App. B.3
eq:app_dp_recurrence .. eq:app_terminal_predecessor) and the stabilised
curvature and boundary score (App. B.2 eq:app_stabilized_curvature,
eq:app_boundary_score) at sampled positions.  Calls only the oracle and the
seeded input generator (hidden states and surprisal generated on the CPU).

    python tests/golden/make_segment_golden.py [config ...]
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import gracekv_oracle as O  # noqa: E402
from synth.workloads import CONFIGS, make_hidden, make_surprisal, segment_starts  # noqa: E402

N_SAMPLES = 96


def sample_positions(T: int) -> np.ndarray:
    """Every position class: the window edges (zeros of the curvature), the
    interior, the end."""
    rng = np.random.default_rng(20261202)
    edge = [0, 1, 3, 4, 15, 16, 17, T - 17, T - 16, T - 1]
    return np.unique(np.concatenate([edge, rng.integers(0, T, N_SAMPLES - len(edge))]))


def main(names):
    for name in names:
        sh = CONFIGS[name]
        st = segment_starts(sh, 0)
        h = make_hidden(sh, 0, st, "cpu").float().numpy().astype(np.float64)
        s = make_surprisal(sh, 0, st, "cpu").numpy()
        bud = O.budget(sh.L, sh.G, sh.N_ctx, sh.x)
        seg = O.segment(h, s, bud.N_c)
        pos = sample_positions(sh.T)
        path = os.path.join(HERE, f"segment_{name}.txt")
        with open(path, "w") as fh:
            fh.write(f"# Oracle segmentation of the {name} workload, seed 0 (hidden states and surprisal\n"
                     f"# from the seeded generator on the CPU), written by make_segment_golden.py.\n"
                     f"# N_c {bud.N_c}, J {len(seg.slot_starts)}.\n")
            fh.write("slots " + " ".join(str(a) for a in seg.slot_starts) + "\n")
            fh.write("pos " + " ".join(str(int(i)) for i in pos) + "\n")
            fh.write("kappa " + " ".join(f"{seg.kappa[i]:.12e}" for i in pos) + "\n")
            fh.write("b " + " ".join(f"{seg.b[i]:.12e}" for i in pos) + "\n")
        print(path, len(seg.slot_starts), flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or ["8b-8k", "8b-32k"])
