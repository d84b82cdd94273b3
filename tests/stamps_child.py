"""Child process of tests/test_gpu_stamps.py: loads the diagnostic build (the parent sets
VIDEOMLA_LIBRARY=stamps), runs tests/stamps_run.py with a stamp buffer attached, checks the
records and saves the outputs for the parent to compare. Usage: stamps_child.py OUT_DIR."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

import paper_2605_30351_amd as vm  # noqa: E402
from tests.stamps_run import run  # noqa: E402

# Expected grids at the Wan shape on a 256-CU device (each launcher's own arithmetic):
# packed write ceil(4680 / ceil(4680 / 256)) = 247 workgroups of 7 waves (224 outputs / 32);
# wide write at batch 4: ceil(18720 / ceil(18720 / 256)) = 253 of 7 compute waves + 1 loader;
# q_absorb 37 token blocks x 12 heads of 4 waves; latent_attend 256 of 8 waves; out_proj
# 19 token blocks x 12 heads of 8 waves.
EXPECT = {  # kernel: (workgroups, waves, points in the order they are reached)
    "cache_write_packed": (247, 7, [0, 1, 2, 3, 4, 5, 6]),
    "cache_write_wide": (253, 7, [0, 1] + [2 + p for p in range(8)] + [12, 13, 14, 15]),
    "q_absorb": (444, 4, [0, 1, 2, 3, 4, 5, 6]),
    "latent_attend": (256, 8, [0, 1] + list(range(2, 10)) + [10, 11]),
    "out_proj": (228, 8, [0, 1, 2, 3, 4, 5]),
}


def check(rec, name):
    n_wg, waves, pts = EXPECT[name]
    k = rec[vm.STAMP_KERNEL[name]].astype(np.int64)  # [workgroup][wave][point]
    live = np.nonzero(k[:, :, 0].max(axis=1))[0]
    assert list(live) == list(range(n_wg)), (name, len(live), n_wg)
    seq = k[:n_wg, :waves][:, :, pts]
    assert (seq > 0).all(), (name, "a point was not recorded")
    assert (np.diff(seq, axis=2) >= 0).all(), (name, "points out of order")
    assert (k[:n_wg, waves + (1 if name == "cache_write_wide" else 0):] == 0).all(), name
    if name == "cache_write_wide":  # the loader wave records its start and its end only
        loader = k[:n_wg, waves]
        assert (loader[:, 0] > 0).all() and (loader[:, 15] >= loader[:, 0]).all(), name
        assert (loader[:, 1:15] == 0).all(), name
    if name == "latent_attend":  # workgroups with two segments: the switch, in order
        two = k[:n_wg, :, 14].max(axis=1) > 0
        sw = k[:n_wg][two][:, :waves][:, :, [1, 12, 13, 14, 10, 11]]
        assert two.sum() > 0 and (sw > 0).all() and (np.diff(sw, axis=2) >= 0).all(), name
        one = k[:n_wg][~two][:, :waves]  # one segment: points 12 and 13 follow its last step
        assert (one[:, :, 12] >= one[:, :, 10]).all() and (one[:, :, 13] >= one[:, :, 12]).all(), name
        print(f"latent_attend: {int(two.sum())} workgroups with two segments, switch points in order")
    print(f"{name}: {n_wg} workgroups x {waves} waves, points {pts} recorded in order", flush=True)


def main():
    assert vm.STAMPS, "the parent sets VIDEOMLA_LIBRARY=stamps"
    assert torch.cuda.get_device_properties(0).multi_processor_count == 256
    buf = torch.zeros(vm.stamps_buffer_bytes() // 8, dtype=torch.int64, device="cuda:0")
    outs = run(vm, buf)
    rec = buf.cpu().numpy().view(np.uint64).reshape(
        vm.STAMP_KERNELS, vm.STAMP_WORKGROUPS, vm.STAMP_WAVES, vm.STAMP_POINTS)
    for name in EXPECT:
        check(rec, name)
    for name, t in outs.items():
        np.save(os.path.join(sys.argv[1], name + ".npy"), t.numpy())
    print("stamps child OK", flush=True)


if __name__ == "__main__":
    main()
