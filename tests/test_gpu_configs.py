"""Parity on the five synthetic workloads at their full batch sizes, in the
launch configuration the benchmark times. At input seed 0 every image of every
workload is checked completely against the oracle (stage by stage, then end to
end); seeds 1 and 2 check a sample of images (images are independent, so a
sampled image is checked exactly as in a batch of one). The cosine the argmax
step reports for each chosen neighbour is compared with the oracle's float64
cosine of the same pair, per stage."""
import numpy as np
import pytest
import torch

import paper_2604_05718_amd as mpm
from paper_2604_05718_amd import synth
from parity import check_schedule_image, to_host

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")

# Seeds 1 and 2: a sample of images per workload (for the stress workload, duplicated-patch images included).
SAMPLES_OTHER_SEEDS = {"vit_ti_512": [0], "vit_s_512": [9, 31], "vit_b_512": [0, 47], "vit_l_1024": [7],
                       "stress_768": [5, 12]}
# The argmax's float32 cosine of the chosen pair against the oracle's float64 one. A float32
# sum of D products of bf16 values has a relative error of at most about D * 2^-24 (about
# 6e-5 at D = 1024); the observed errors are two orders of magnitude smaller, and this bound
# keeps them below the near-tie threshold the parity protocol relies on.
BEST_ABS_TOL = 1e-5


def best_error(res, x, cfg, images, reports_by_image):
    """Max |best - oracle cosine| per stage over the given images (rows where the GPU
    chose the oracle's neighbour)."""
    errs = []
    cur, cur_off = x, None
    for s, st in enumerate(res.stages):
        nb, best = mpm.argmax(cur, x_off=cur_off, N=cfg.N, with_best=True)
        torch.cuda.synchronize()
        nb, best = nb.cpu().numpy(), best.cpu().numpy().astype(np.float64)
        e = 0.0
        for b in images:
            nn = reports_by_image[b][s].oracle_nearest
            n = nn.nb.shape[0]
            if n < 2:
                continue
            same = nb[b, :n] == nn.nb
            e = max(e, float(np.max(np.abs(best[b, :n][same] - nn.top1[same]), initial=0.0)))
        errs.append(e)
        cur, cur_off = st.y, st.y_off
    return errs


@pytest.mark.timeout(900)
@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", list(SAMPLES_OTHER_SEEDS))
def test_config_parity(name, seed):
    cfg = synth.config(name)
    print(f"config {name} seed {seed}: B={cfg.B} N={cfg.N} D={cfg.D} {cfg.dtype} insertions={cfg.insertions}",
          flush=True)
    x = synth.make_batch(cfg, seed=seed)
    xd = x.to(DEV)
    res = mpm.run_schedule(xd, insertions=cfg.insertions)
    torch.cuda.synchronize()
    h = to_host(res)
    images = range(cfg.B) if seed == 0 else SAMPLES_OTHER_SEEDS[name]
    reports = {}
    near = [0] * cfg.insertions
    flips = [0] * cfg.insertions
    worst = [0.0] * cfg.insertions
    for b in images:
        reps = check_schedule_image(x[b], cfg.dtype, h, b)
        reports[b] = reps
        for s, r in enumerate(reps):
            near[s] += r.near_tie_rows
            flips[s] += r.flipped_rows
            worst[s] = max(worst[s], r.max_feature_rel_err)
    best = best_error(res, xd, cfg, list(images), reports)
    for s in range(cfg.insertions):
        print(f"  stage {s + 1}: {len(images)} images checked, near-tie rows {near[s]}, accepted flips {flips[s]}, "
              f"max feature rel err {worst[s]:.1e}, max |best - cos| {best[s]:.2e}", flush=True)
    assert max(best) < BEST_ABS_TOL, best
    # Structure of the whole batch (every image): counts within the pairing bounds.
    n_prev = np.full(cfg.B, cfg.N, dtype=np.int64)
    for off in h.y_off:
        cnt = np.diff(off)
        assert np.all(cnt >= (n_prev + 1) // 2) and np.all(cnt <= np.maximum(n_prev - 1, 1))
        n_prev = cnt
