"""The accumulation error of the FP8 score product, measured on the GPU (vc_fp8_score_product runs
the instruction sequence of the attention kernel's FP8 scores: two chained E4M3 32x32x64 matrix
instructions, channels 0..63 then 64..127).

The FP8-QK configuration (Sec. 4.5) takes its scores from the matrix unit, which does not sum the
products of a dot exactly once they span many binades. The attention tolerance of that mode
(reading R23) rests on this bound per instruction: the result differs from the exact sum of the
accumulator input and the products by at most E = 2^-10.5 times the larger of the largest
product magnitude and the accumulator input's magnitude. Chained over the two instructions of a
score that gives

    |score - exact| <= E (2 max(max|product|, |c_in|) + |c_in + sum of the first 64 products|)
                       + 2^-23 |exact|                                 (the result is an fp32)

which is the `eps` that the FP8-QK parity tests (test_gpu_fp8qk.flip_bound and
test_gpu_codes.f8_expcast_window) propagate into the probability codes. This file checks that
bound on seeded E4M3 operands spanning the whole exponent range, on operands shaped like the
rotated, block-scaled Q/K codes, with and without a large accumulator input; and that products
confined to a narrow exponent window are summed exactly (the premise of
test_gpu_fp8qk.test_forward_f8_exact_window).
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
vc = pytest.importorskip("paper_2609_15810_amd")

pytestmark = pytest.mark.gpu

E = 2.0 ** -10.5          # the per-instruction bound the FP8-QK tolerance assumes
NBLK = 256


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    vc.lib()


def dec(b):
    return torch.from_numpy(np.ascontiguousarray(b, np.uint8)).view(torch.float8_e4m3fn).double().numpy()


def enc(x):
    """E4M3 bytes of fp32 values |x| <= 448 (the library's nearest-even cast)."""
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def full_range(rng):
    """Uniform over every finite E4M3 byte (subnormals and both signs included)."""
    codes = np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8)
    return rng.choice(codes, (NBLK, 32, 128)).astype(np.uint8)


def rotated(rng):
    """Rows like the prepared Q/K codes: Gaussian rows with two outlier channels x10, rotated by the
    128-point Hadamard matrix, scaled so that each 32-row block's largest magnitude is 448."""
    from scipy.linalg import hadamard
    x = rng.standard_normal((NBLK, 32, 128))
    x[:, :, rng.choice(128, 2, replace=False)] *= 10.0
    x = x @ hadamard(128).astype(np.float64)
    x *= 448.0 / np.abs(x).max(axis=(1, 2), keepdims=True)
    return enc(x.astype(np.float32))


def narrow(rng):
    """Magnitudes within a factor 4 (random signs): every product lies within a factor 16."""
    x = rng.choice([-1.0, 1.0], (NBLK, 32, 128)) * rng.uniform(0.25, 1.0, (NBLK, 32, 128)) * 3.0
    return enc(x.astype(np.float32))


def run(a, b, c_in):
    dev = lambda t, dt: torch.from_numpy(np.ascontiguousarray(t, dt)).cuda()
    out = torch.empty((a.shape[0], 32, 32), dtype=torch.float32, device="cuda")
    vc.vc_fp8_score_product(dev(a, np.uint8), dev(b, np.uint8), dev(c_in, np.float32), out)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def exact_parts(a, b, c_in):
    """Exact (fp64) products [n, 32, 32, 128], the exact result and the exact first partial."""
    da, db = dec(a), dec(b)
    prod = da[:, :, None, :] * db[:, None, :, :]
    first = c_in + prod[..., :64].sum(axis=-1)
    return prod, first + prod[..., 64:].sum(axis=-1), first


@pytest.mark.parametrize("kind", ["full_range", "rotated"])
@pytest.mark.parametrize("acc", ["zero", "large"])
def test_fp8_product_error_bound(kind, acc):
    rng = np.random.default_rng({"full_range": 1, "rotated": 2}[kind] * 10 + (acc == "large"))
    gen = {"full_range": full_range, "rotated": rotated}[kind]
    a, b = gen(rng), gen(rng)
    c_in = np.zeros((NBLK, 32, 32))
    if acc == "large":
        prod, _, _ = exact_parts(a, b, c_in)
        scale = np.abs(prod).max(axis=-1)
        c_in = (rng.choice([-1.0, 1.0], scale.shape) * scale * 2.0 ** rng.uniform(-4, 6, scale.shape))
        c_in = c_in.astype(np.float32).astype(np.float64)
    out = run(a, b, c_in)
    prod, exact, first = exact_parts(a, b, c_in)
    err = np.abs(out - exact)
    pm1 = np.maximum(np.abs(prod[..., :64]).max(axis=-1), np.abs(c_in))
    pm2 = np.maximum(np.abs(prod[..., 64:]).max(axis=-1), np.abs(first))
    scale1 = np.maximum(np.abs(prod).max(axis=-1), np.abs(c_in))
    bound = E * (2 * scale1 + np.abs(first)) * (1 + 2 * E) + np.abs(exact) * 2.0 ** -23 + 2.0 ** -140
    ratio = err / np.maximum(pm1 + pm2, 1e-300)
    inexact = float((err > np.abs(exact) * 2.0 ** -23).mean())
    print(f"{kind}/{acc}: {inexact:.3f} of scores inexact, worst error {np.log2(ratio.max() + 1e-300):.2f} "
          f"(log2, relative to the sum of both instructions' scales), worst against the bound "
          f"{(err / bound).max():.3f}")
    assert (err <= bound).all(), np.unravel_index(np.argmax(err / bound), err.shape)


def test_fp8_product_exact_in_narrow_window():
    rng = np.random.default_rng(5)
    a, b = narrow(rng), narrow(rng)
    c_in = np.zeros((NBLK, 32, 32))
    out = run(a, b, c_in)
    _, exact, _ = exact_parts(a, b, c_in)
    # every value is a multiple of 2^-4 of magnitude <= 3, so the exact sum is a multiple of 2^-8
    # below 2^11: representable in fp32
    assert np.array_equal(out, exact)
