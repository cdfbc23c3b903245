"""Un-tiling of the library's code layouts (as documented in include/vc_attn.h) for comparison
with the oracle's logical [row, channel] arrays. Pure index bookkeeping, no arithmetic."""
import numpy as np


def _qk_index():
    row = np.arange(128)[:, None]
    ch = np.arange(128)[None, :]
    return (((row // 32) * 4 + ch // 32) * 2 + (ch % 32) // 16) * 512 + (row % 32) * 16 + ch % 16


def _v_index():
    key = np.arange(128)[:, None]
    ch = np.arange(128)[None, :]
    kb, w = key // 32, key % 32
    kc, sh, kh, t = kb // 2, kb % 2, (w % 8) // 4, 4 * (w // 8) + w % 4
    return ((((kc * 4 + ch // 32) * 2 + kh) * 2 + sh) * 32 + ch % 32) * 16 + t


QK_INDEX = _qk_index()
V_INDEX = _v_index()


def untile(phys: np.ndarray, index: np.ndarray) -> np.ndarray:
    """phys: [..., Np, 128] tiled bytes -> logical [..., Np, 128]."""
    shp = phys.shape
    blocks = phys.reshape(-1, 128 * 128)
    out = blocks[:, index.reshape(-1)].reshape(-1, 128, 128)
    return out.reshape(shp)


def untile_qk(phys):
    return untile(phys, QK_INDEX)


def untile_v(phys):
    return untile(phys, V_INDEX)
