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


def _mx_code_index():
    """byte index and nibble shift of channel ch of row `row` in a packed MXFP4 block:
    [rb 4][m 2][h 2][r 32][16 bytes], two channels per byte (even channel in the low nibble)."""
    row = np.arange(128)[:, None]
    ch = np.arange(128)[None, :]
    rb, r, m, h = row // 32, row % 32, ch // 64, (ch % 64) // 32
    byte = ((rb * 2 + m) * 2 + h) * 512 + r * 16 + (ch % 32) // 2
    return byte, np.broadcast_to(4 * (ch % 2), byte.shape)


def _mx_scale_index():
    """position of the E8M0 byte of row `row`, 32-channel block b (b = 2m + h) in the 512 scale
    bytes of a block: [lane 64][rb 4][m 2] with lane = 32h + r."""
    row = np.arange(128)[:, None]
    b = np.arange(4)[None, :]
    rb, r, m, h = row // 32, row % 32, b // 2, b % 2
    return (h * 32 + r) * 8 + rb * 2 + m


MX_CODE_BYTE, MX_CODE_SHIFT = _mx_code_index()
MX_SCALE_INDEX = _mx_scale_index()


def untile_mx_codes(phys: np.ndarray) -> np.ndarray:
    """phys: [..., Np, 64] packed bytes -> one E2M1 code per byte [..., Np, 128]."""
    shp = phys.shape
    blocks = phys.reshape(-1, 128 * 64).astype(np.uint8)
    out = (blocks[:, MX_CODE_BYTE.reshape(-1)] >> MX_CODE_SHIFT.reshape(-1).astype(np.uint8)) & 15
    return out.reshape(shp[:-1] + (128,))


def untile_mx_scales(phys: np.ndarray) -> np.ndarray:
    """phys: [..., Np, 4] scale bytes in the library's order -> [..., Np, 4] by (row, block)."""
    shp = phys.shape
    blocks = phys.reshape(-1, 128 * 4).astype(np.uint8)
    return blocks[:, MX_SCALE_INDEX.reshape(-1)].reshape(shp)


def _f8_index():
    """FP8 Q/K block layout [rb 4][m 2][h 2][half 2][r 32][e 16]: lane h*32 + r of the FP8
    32x32x64 product holds channels 64m + 32h .. + 31 of row 32rb + r as two 16-byte halves."""
    row = np.arange(128)[:, None]
    ch = np.arange(128)[None, :]
    rb, r, m, h, half, e = row // 32, row % 32, ch // 64, (ch % 64) // 32, (ch % 32) // 16, ch % 16
    return ((((rb * 2 + m) * 2 + h) * 2 + half) * 32 + r) * 16 + e


F8_INDEX = _f8_index()


def untile_f8(phys):
    return untile(phys, F8_INDEX)
