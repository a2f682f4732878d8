"""Helpers for the GPU tests: device buffers, calls through the C-ABI, and host-side
unpacking of the blocked transform-domain layouts documented in include/wino.h."""
import numpy as np
import torch

from paper_1903_01521_amd import binding as B

DEV = "cuda:0"


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def geometry(N, H, W, pad, m):
    Ho, Wo = H + 2 * pad - 2, W + 2 * pad - 2
    th, tw = -(-Ho // m), -(-Wo // m)
    return Ho, Wo, th, tw, N * th * tw


def empty_bytes(nbytes: int, fill=float("nan")) -> torch.Tensor:
    return torch.full((max(nbytes // 4, 1),), fill, dtype=torch.float32, device=DEV)


def filter_transform(g: np.ndarray, m: int) -> torch.Tensor:
    K, C = g.shape[:2]
    U = empty_bytes(B.wino_filter_bytes(C, K, m))
    B.check(B.wino_filter_transform(dev(g), U, C, K, m), "wino_filter_transform")
    return U


def conv2d(x, U, K, pad, m, flags=0, y=None):
    """y = layer(x) through wino_conv2d; x may be numpy or a device tensor."""
    xt = dev(x) if isinstance(x, np.ndarray) else x
    N, C, H, W = xt.shape
    Ho, Wo, *_ = geometry(N, H, W, pad, m)
    if y is None:
        y = torch.full((N, K, Ho, Wo), float("nan"), dtype=torch.float32, device=DEV)
    wsb = B.wino_workspace_bytes(N, C, H, W, K, pad, m, flags)
    assert wsb != 2**64 - 1
    ws = empty_bytes(wsb) if wsb else None
    B.check(B.wino_conv2d(xt, U, y, N, C, H, W, K, pad, m, flags, ws, wsb), "wino_conv2d")
    return y


def input_transform(x, pad, m):
    xt = dev(x) if isinstance(x, np.ndarray) else x
    N, C, H, W = xt.shape
    V = empty_bytes(B.wino_input_tf_bytes(N, C, H, W, pad, m))
    B.check(B.wino_input_transform(xt, V, N, C, H, W, pad, m), "wino_input_transform")
    return V


def batched_gemm(U, V, N, C, H, W, K, pad, m):
    M = empty_bytes(B.wino_gemm_out_bytes(N, K, H, W, pad, m))
    B.check(B.wino_batched_gemm(U, V, M, N, C, H, W, K, pad, m), "wino_batched_gemm")
    return M


def output_transform(M, N, K, H, W, pad, m, flags=0):
    Ho, Wo, *_ = geometry(N, H, W, pad, m)
    y = torch.full((N, K, Ho, Wo), float("nan"), dtype=torch.float32, device=DEV)
    B.check(B.wino_output_transform(M, y, N, K, H, W, pad, m, flags), "wino_output_transform")
    return y


# ---- layout unpacking (host side, from the documented layouts) ----------------

def _pad_counts(C, K, P):
    CQ, KB, PB = -(-C // 4), -(-K // 16), -(-P // 16)
    return CQ, KB, PB


def unpack_U(U: np.ndarray, C: int, K: int, m: int, crop=True, r: int = 3) -> np.ndarray:
    """U[KB][CQ][T/4][64][4] (lane = (c%4)*16 + k%16, slot t%4) -> logical [T][C][K]."""
    T = (m + r - 1) ** 2
    CQ, KB, _ = _pad_counts(C, K, 1)
    a = U[:KB * CQ * T * 64].reshape(KB, CQ, T // 4, 4, 16, 4)           # kb, cq, tg, cl, kl, tt
    a = a.transpose(2, 5, 1, 3, 0, 4).reshape(T, CQ * 4, KB * 16)        # t, c, k
    return a[:, :C, :K] if crop else a


def unpack_V(V: np.ndarray, C: int, P: int, m: int, crop=True) -> np.ndarray:
    """V[PB][CQ][T/4][64][4] (lane = (c%4)*16 + p%16, slot t%4) -> logical [T][C][P]."""
    T = (m + 2) ** 2
    CQ, _, PB = _pad_counts(C, 1, P)
    a = V[:PB * CQ * T * 64].reshape(PB, CQ, T // 4, 4, 16, 4)           # pb, cq, tg, cl, pl, tt
    a = a.transpose(2, 5, 1, 3, 0, 4).reshape(T, CQ * 4, PB * 16)        # t, c, p
    return a[:, :C, :P] if crop else a


def unpack_M(M: np.ndarray, K: int, P: int, m: int, crop=True) -> np.ndarray:
    """M[PB][KB][T][64][4] (lane = 16*((k%16)/4) + p%16, slot k%4) -> logical [T][K][P]."""
    T = (m + 2) ** 2
    _, KB, PB = _pad_counts(1, K, P)
    a = M[:PB * KB * T * 256].reshape(PB, KB, T, 4, 16, 4)       # pb, kb, t, kq, pl, r
    a = a.transpose(2, 1, 3, 5, 0, 4).reshape(T, KB * 16, PB * 16)
    return a[:, :K, :P] if crop else a


def pack_M(Ml: np.ndarray, K: int, P: int, m: int) -> np.ndarray:
    """Inverse of unpack_M for a logical [T][K][P] array (padding filled with 0)."""
    T = (m + 2) ** 2
    _, KB, PB = _pad_counts(1, K, P)
    full = np.zeros((T, KB * 16, PB * 16), dtype=np.float32)
    full[:, :K, :P] = Ml
    a = full.reshape(T, KB, 4, 4, PB, 16)                         # t, kb, kq, r, pb, pl
    return np.ascontiguousarray(a.transpose(4, 1, 0, 2, 5, 3)).reshape(-1)


def normwise_err(y: np.ndarray, ref: np.ndarray) -> float:
    """max |y - ref| / max |ref| over the whole tensor."""
    return float(np.abs(y.astype(np.float64) - ref).max() / max(np.abs(ref).max(), 1e-300))
