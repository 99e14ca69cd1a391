"""Parity on the five synthetic workloads at their full batch sizes, in the
launch configuration the benchmark times, for input seeds 0, 1 and 2. The GPU
runs every image; the oracle checks a sample of images completely (images are
independent, so a sampled image is checked exactly as in a batch of one)."""
import pytest
import torch

import paper_2604_05718_amd as mpm
from paper_2604_05718_amd import synth
from parity import check_schedule_image

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")

SAMPLES = {
    "vit_ti_512": [0],
    "vit_s_512": [0, 17, 31],
    "vit_b_512": [0, 33, 63],
    "vit_l_1024": [0, 15],
    "stress_768": [5, 12, 25],   # 5 and 25 are duplicated-patch images
}
# Seeds 1 and 2 check one image per workload (for the stress workload a duplicated-patch one).
SAMPLES_OTHER_SEEDS = {"vit_ti_512": [0], "vit_s_512": [9], "vit_b_512": [47], "vit_l_1024": [7], "stress_768": [15]}


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("name", list(SAMPLES))
def test_config_parity(name, seed):
    cfg = synth.config(name)
    print(f"config {name} seed {seed}: B={cfg.B} N={cfg.N} D={cfg.D} {cfg.dtype} insertions={cfg.insertions}",
          flush=True)
    x = synth.make_batch(cfg, seed=seed)
    res = mpm.run_schedule(x.to(DEV), insertions=cfg.insertions)
    torch.cuda.synchronize()
    for b in (SAMPLES if seed == 0 else SAMPLES_OTHER_SEEDS)[name]:
        reps = check_schedule_image(x[b], cfg.dtype, res, b)
        summary = ", ".join(
            f"stage{s + 1}: n={r.n} n'={r.count} near-tie rows={r.near_tie_rows} accepted flips={r.flipped_rows} "
            f"max rel err={r.max_feature_rel_err:.1e}" for s, r in enumerate(reps))
        print(f"  image {b}: {summary}", flush=True)
    # Structure of the whole batch (every image): counts within the pairing bounds.
    n_prev = torch.full((cfg.B,), cfg.N, dtype=torch.int64)
    for st in res.stages:
        cnt = torch.diff(st.y_off.cpu().to(torch.int64))
        assert torch.all(cnt >= (n_prev + 1) // 2) and torch.all(cnt <= torch.clamp(n_prev - 1, min=1))
        n_prev = cnt
