"""One Wan2.1-1.3B chunk-step and one batch-4 cache write, run identically by the GPU test of
the diagnostic build (tests/test_gpu_stamps.py) in its own process with the product library
and, through tests/stamps_child.py, in a child process with the diagnostic build. Inputs are
drawn on the GPU from a seeded generator, so both processes see the same values."""
import torch

from workloads import WAN


def run(vm, stamp_buffer=None):
    """Ring fill of 21 frames, then the chunk-step at frame 21 (packed cache write and the
    attend on the even split) and a batch-4 cache write of the same frames. With
    `stamp_buffer` the two steps record into it (diagnostic build only). Returns the outputs as
    int16 tensors on the host."""
    d, dev = WAN, torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(2605)

    def normal(shape, std=1.0):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    nq, H = d.chunk_tokens, d.n_heads
    w_dkv = normal((d.d_c, d.d_model), d.d_model ** -0.5)
    w_kr = normal((d.d_rope, d.d_model), d.d_model ** -0.5)
    w_uk = normal((H * d.d_nope, d.d_c), d.d_c ** -0.5)
    w_uv = normal((H * d.d_v, d.d_c), d.d_c ** -0.5)
    gamma = (1 + 0.1 * normal((d.d_c,))).to(torch.bfloat16)
    w_packed = torch.empty(vm.write_weights_bytes(d), dtype=torch.uint8, device=dev)
    vm.prepare_write_weights(d, w_dkv, w_kr, w_packed)
    c_kv = torch.zeros((1, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k_r = torch.zeros((1, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    for f in range(0, d.window_frames, d.chunk_frames):
        vm.cache_write_prepared(d, f, 1, normal((1, nq, d.d_model)), w_packed, gamma, c_kv, k_r)
    fe = d.window_frames
    x = normal((1, nq, d.d_model))
    q_nope, q_r = normal((1, nq, H, d.d_nope)), normal((1, nq, H, d.d_rope))
    out = torch.empty((1, nq, H, d.d_v), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(vm.attend_workspace_bytes(d, 1), dtype=torch.uint8, device=dev)
    x4 = normal((4, nq, d.d_model))
    c4 = torch.zeros((4, d.window_tokens, d.d_c), dtype=torch.bfloat16, device=dev)
    k4 = torch.zeros((4, d.window_tokens, d.d_rope), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    if stamp_buffer is not None:
        vm.stamps_attach(stamp_buffer)
    try:
        vm.cache_write_prepared(d, fe, 1, x, w_packed, gamma, c_kv, k_r)
        vm.attend(d, fe, 1, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws,
                  opts=vm.AttendOpts(partition="even"))
        vm.cache_write_prepared(d, fe, 4, x4, w_packed, gamma, c4, k4)
        torch.cuda.synchronize()
    finally:
        if stamp_buffer is not None:
            vm.stamps_attach(None)
    return {name: t.view(torch.int16).cpu() for name, t in
            (("c_kv", c_kv), ("k_r", k_r), ("out", out), ("c_kv_b4", c4), ("k_r_b4", k4))}
