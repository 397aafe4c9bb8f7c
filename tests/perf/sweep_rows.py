"""Row lists of one PatchMatch sweep, from the oracle's candidate trace (a measurement aid).

For every query of the 256x256 bf16 workload (4 slices, d = 64), the key rows that sweep t of
Algorithm 1 reads, in the order the sweep kernel reads them: first the propagation candidates
and random-search step 0 that lie inside the key grid and differ from the incumbent, then
random-search steps 1, 2, ... (each around the running best).  The maps J_0 .. J_{t-1} come from
the oracle.  Writes ``rows_t<t>.bin`` (int32 [n, 32], slice-local key rows, -1 padded) and
``cnt_t<t>.bin`` (int32 [n]) into OUTDIR for ``gather_replay``.

    python tests/perf/sweep_rows.py OUTDIR [t]
"""
import os
import sys
import time

import numpy as np

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "..", ".."))
import oracle  # noqa: E402
import scram_inputs as si  # noqa: E402

MAXR = 32


def main():
    out = sys.argv[1]
    t = int(sys.argv[2]) if len(sys.argv) > 2 else 4
    os.makedirs(out, exist_ok=True)
    cfg = si.get(si.HEADLINE)
    a = si.make_arrays(cfg)
    Q, K = a["Q"].astype(np.float64), a["K"].astype(np.float64)
    J, _ = oracle.pm_init(Q, K, cfg.pm_seed)
    for k in range(1, t):
        J = oracle.patchmatch(Q, K, 1, cfg.pm_seed, init=J, t0=k)[0]
    s_prev, _ = oracle.pm_scores(Q, K, J)
    n = J.size
    Jf = J.reshape(-1)
    rows = np.full((n, MAXR), -1, np.int32)
    cnt = np.zeros(n, np.int32)
    t0 = time.time()
    for g in range(n):
        idx, kind, _, _ = oracle.pm_trace(Q, K, J, t, cfg.pm_seed, g, cap=64, s_prev=s_prev)
        # stage 1 drops candidates equal to the incumbent; random-search steps >= 1 are always read
        keep = [int(i) for i, kd in zip(idx, kind) if kd > 100 or i != Jf[g]]
        cnt[g] = len(keep)
        rows[g, :len(keep)] = keep
        if g % 65536 == 0:
            print(f"traced {g} of {n} queries ({time.time() - t0:.0f} s)", flush=True)
    rows.tofile(os.path.join(out, f"rows_t{t}.bin"))
    cnt.tofile(os.path.join(out, f"cnt_t{t}.bin"))
    print(f"sweep {t}: {cnt.mean():.2f} key rows per query (max {cnt.max()})", flush=True)


if __name__ == "__main__":
    main()
