"""Helpers of the GPU parity tests: move a workload to the GPU, run, compare."""
import dataclasses

import numpy as np
import torch

import paper_2606_16824_amd as cwlib

BF16_MAX_ABS, BF16_MEAN_ABS = 2e-2, 2e-3  # bf16 pool, N(0,1) inputs
FP8_MAX_ABS = 6e-2  # fp8 pool, against the oracle on the same dequantised values


@dataclasses.dataclass
class DeviceWorkload:
    q: torch.Tensor
    k_new: torch.Tensor
    v_new: torch.Tensor
    k_pool: torch.Tensor
    v_pool: torch.Tensor
    k_scale: object
    v_scale: object
    block_table: torch.Tensor
    spec: object


def to_gpu(w, device="cuda:0") -> DeviceWorkload:
    mv = lambda t: None if t is None else t.to(device).contiguous()
    return DeviceWorkload(mv(w.q), mv(w.k_new), mv(w.v_new), mv(w.k_pool), mv(w.v_pool),
                          mv(w.k_scale), mv(w.v_scale), mv(w.block_table), w.spec)


def run_extend(dw: DeviceWorkload, with_lse=True, workspace=None):
    s = dw.spec
    lse = torch.full((dw.q.shape[0], dw.q.shape[1]), float("nan"), device=dw.q.device) if with_lse else None
    out = torch.full_like(dw.q, float("nan"))
    cwlib.extend_attention(dw.q, dw.k_new, dw.v_new, dw.k_pool, dw.v_pool, dw.block_table,
                           s.prefix_lens, s.suffix_lens, s.gqa_group, s.softmax_scale,
                           k_scale=dw.k_scale, v_scale=dw.v_scale, out=out, lse=lse,
                           workspace=workspace)
    torch.cuda.synchronize()
    return out, lse


def bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def as_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().to(torch.float64).numpy()


# every comparison of the session, (what, n, max_abs, bound, mean_abs, bound), printed
# as one table at the end of the run (tests/conftest.py) so the headroom shows
MARGINS = []


def assert_close(got: np.ndarray, ref: np.ndarray, max_abs: float, mean_abs: float = None, what=""):
    assert got.shape == ref.shape, (got.shape, ref.shape)
    bad = ~np.isfinite(got)
    if bad.any():
        idx = np.argwhere(bad)
        print(f"[{what}] {int(bad.sum())} non-finite values; first indices {idx[:12].tolist()}; "
              f"rows with any: {np.unique(idx[:, 0]).tolist()[:40]}", flush=True)
    assert not bad.any(), f"{what}: non-finite GPU output"
    err = np.abs(got - ref)
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    print(f"[{what}] max_abs={mx:.3e} mean_abs={mean:.3e} n={err.size}", flush=True)
    MARGINS.append((what, int(err.size), mx, max_abs, mean, mean_abs))
    assert mx <= max_abs, f"{what}: max abs error {mx:.3e} > {max_abs:.1e}"
    if mean_abs is not None:
        assert mean <= mean_abs, f"{what}: mean abs error {mean:.3e} > {mean_abs:.1e}"
    return mx, mean


def assert_within_bf16_ulps(got: np.ndarray, ref: np.ndarray, ulps: int = 2, what=""):
    """Two bf16 results of the same quantity computed in different orders (another
    split of the keys, another kernel): |got - ref| <= `ulps` bf16 ulps of the larger
    magnitude, taken at least at 0.5 (so values below 1 get 2^-7 with ulps = 2)."""
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite GPU output"
    mag = np.maximum(np.maximum(np.abs(got), np.abs(ref)), 0.5)
    bound = ulps * np.exp2(np.floor(np.log2(mag)) - 7)  # bf16 keeps 8 significant bits
    ratio = np.abs(got - ref) / bound
    worst = float(ratio.max()) if ratio.size else 0.0
    err = np.abs(got - ref)
    print(f"[{what}] max_abs={float(err.max()) if err.size else 0.0:.3e} "
          f"worst {worst:.2f} of {ulps} ulps n={err.size}", flush=True)
    MARGINS.append((what + f" (in units of {ulps} bf16 ulps)", int(err.size), worst, 1.0,
                    float(err.mean()) if err.size else 0.0, None))
    assert worst <= 1.0, f"{what}: difference above {ulps} bf16 ulps (worst {worst:.2f})"
