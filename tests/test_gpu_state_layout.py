"""The state's tile-major layout: sketchssm_state_to_tiles and
sketchssm_state_from_tiles against a plain torch permutation written from the
layout's definition (tile (vt, kt) of 16 x 16 at (vt * K/16 + kt) * 256,
element X[16 vt + r][16 kt + c] at 4 (r + 16 (c / 4)) + c % 4), and their
round trip.  Bitwise: the conversion moves floats and computes nothing."""
import pytest
import torch

from paper_2609_33051_amd import binding as B

pytestmark = pytest.mark.gpu


def tiles_reference(X):
    """X [B][H][V][K] -> [B][H][V*K] tile-major, by definition."""
    Bt, H, V, K = X.shape
    t = X.reshape(Bt, H, V // 16, 16, K // 16, 4, 4)          # b h vt r kt cg ci
    return t.permute(0, 1, 2, 4, 5, 3, 6).reshape(Bt, H, V * K)  # b h vt kt cg r ci


@pytest.mark.parametrize("Bt,H,K,V", [(3, 2, 64, 64), (2, 5, 128, 64), (4, 3, 128, 128), (1, 1, 128, 128)])
def test_state_layout_matches_definition(Bt, H, K, V):
    print(f"[case] state layout B={Bt} H={H} K={K} V={V}", flush=True)
    cfg = B.make_config("gdn", Bt, H, K, V, 16, 8, "bf16")
    g = torch.Generator(device="cuda").manual_seed(Bt * 1000 + H * 10 + K + V)
    X = torch.randn((Bt, H, V, K), device="cuda", generator=g)
    T = torch.full((Bt, H, V * K), float("nan"), device="cuda")
    B.sketchssm_state_to_tiles(cfg, X, T)
    back = torch.full_like(X, float("nan"))
    B.sketchssm_state_from_tiles(cfg, T, back)
    torch.cuda.synchronize()
    assert torch.equal(T, tiles_reference(X))
    assert torch.equal(back, X)


def test_state_layout_large_grid():
    """More float4s than one pass of the launch grid covers (grid-stride loop)."""
    Bt, H, K, V = 64, 32, 128, 128          # 2^25 floats: 8.4M float4s over at most 16384 x 256 threads
    print(f"[case] state layout grid-stride B={Bt} H={H}", flush=True)
    cfg = B.make_config("kda", Bt, H, K, V, 16, 16, "bf16")
    X = torch.randn((Bt, H, V, K), device="cuda", generator=torch.Generator(device="cuda").manual_seed(5))
    T = torch.empty((Bt, H, V * K), device="cuda")
    B.sketchssm_state_to_tiles(cfg, X, T)
    torch.cuda.synchronize()
    assert torch.equal(T, tiles_reference(X))
