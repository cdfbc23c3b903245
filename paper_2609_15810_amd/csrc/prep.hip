// Fused preprocessing of the 8-bit VC-Attention operands (Sec. 3.4 and Appendix B).
//
// Three launches per call:
//   prep_stats    grid (ceil(T/4), B*H, 2), one wave for four blocks. z = 0: value rows of
//                 permuted block j (gathered by perm), one pass: the block mean mu_j, stored as
//                 bf16, and the per-channel max |V' - mu_j| of the block. z = 1: rotated key
//                 rows of original-order block j summed per channel (the centering statistics).
//   prep_finalize grid (B*H, 16), 256 threads: key channel mean and per-channel value scale.
//   prep_quant    grid (T, B*H, 3), 256 threads. z = 0: K' rows (gather, RoPE, centering,
//                 Hadamard, per-block INT8 or E4M3, or MXFP4); z = 1: V' rows (gather, demean,
//                 per-channel E4M3), transposed into the tile order of the attention kernel;
//                 z = 2: Q rows (RoPE, Hadamard, per-block INT8 or E4M3, or MXFP4).
// All floating-point steps that decide a stored code are written as single IEEE fp32
// operations in a fixed order (compiled with -ffp-contract=off; fused multiply-adds are spelled
// out), so the codes, scales and means are reproducible bit for bit.
#include <type_traits>

#include "vc_common.hpp"
#include "vc_internal.hpp"

namespace vc {

// n / d for 0 <= n < 2^24 and d >= 1: a float estimate, then one correction each way (the
// estimate is within one of the quotient).
__device__ __forceinline__ int div_small(int n, int d, float inv_d) {
  int q = (int)((float)n * inv_d);
  q -= (q * d > n) ? 1 : 0;
  q += ((q + 1) * d <= n) ? 1 : 0;
  return q;
}

// Rows of the rotary tables for token n: frames axis f, rows axis F + y, columns axis F + Ht + x
// (token n = (f * Ht + y) * Wd + x).
struct RopeRows {
  int f, y, x;
};
__device__ __forceinline__ RopeRows rope_rows(int n, const PrepArgs& a) {
  int f, rem, y;
  if (a.N <= (1 << 24)) {
    f = div_small(n, a.Ht * a.Wd, a.inv_hw);
    rem = n - f * (a.Ht * a.Wd);
    y = div_small(rem, a.Wd, a.inv_w);
  } else {
    f = n / (a.Ht * a.Wd);
    rem = n - f * (a.Ht * a.Wd);
    y = rem / a.Wd;
  }
  return RopeRows{f, a.F + y, a.F + a.Ht + (rem - y * a.Wd)};
}

// One rotary pair with the table row of its axis: y0 = fma(x0, c, -(x1 s)), y1 = fma(x0, s, x1 c).
__device__ __forceinline__ void rope_pair(float& x0, float& x1, int pair, const RopeRows& rr, const PrepArgs& a) {
  const int ax = rope_axis(pair);
  const int row = ax == 0 ? rr.f : (ax == 1 ? rr.y : rr.x);
  const float c = a.rope_cos[row * 64 + pair], s = a.rope_sin[row * 64 + pair];
  const float p = x1 * s, q = x1 * c;
  const float y0 = __builtin_fmaf(x0, c, -p);
  const float y1 = __builtin_fmaf(x0, s, q);
  x0 = y0;
  x1 = y1;
}

// ------------------------------------------------------------------------------------------
// Statistics: per-block key channel sums and value block means / residual maxima.
// A wave takes four consecutive blocks, one per 16-lane row of the wave: lane q of a row owns
// channels 8q .. 8q + 7 (rotary pairs 4q .. 4q + 3) and walks its block's rows in ascending
// order with 16-byte loads, so every per-channel sum is a sequential fp32 sum from 0.
// ------------------------------------------------------------------------------------------

// Value v of lane L of the lane's 16-lane row (DPP row_newbcast), L known at compile time.
template <int L>
__device__ __forceinline__ int row_bcast(int v) {
  return __builtin_amdgcn_update_dpp(0, v, 0x150 + L, 0xf, 0xf, false);
}
__device__ __forceinline__ int row_bcast_n(int v, int l) {
  switch (l & 15) {
    case 0: return row_bcast<0>(v);
    case 1: return row_bcast<1>(v);
    case 2: return row_bcast<2>(v);
    case 3: return row_bcast<3>(v);
    case 4: return row_bcast<4>(v);
    case 5: return row_bcast<5>(v);
    case 6: return row_bcast<6>(v);
    case 7: return row_bcast<7>(v);
    case 8: return row_bcast<8>(v);
    case 9: return row_bcast<9>(v);
    case 10: return row_bcast<10>(v);
    case 11: return row_bcast<11>(v);
    case 12: return row_bcast<12>(v);
    case 13: return row_bcast<13>(v);
    case 14: return row_bcast<14>(v);
    default: return row_bcast<15>(v);
  }
}

__device__ __forceinline__ void unpack8(const u4& w, float (&x)[8]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    x[2 * k] = bf16_lo(w[k]);
    x[2 * k + 1] = bf16_hi(w[k]);
  }
}

// Key statistics of block j (original order): rows r0 .. r0 + valid - 1, rotated, summed per
// channel. The rotary table entries of lane q's pairs 4q .. 4q + 3 come as float4 loads from
// the row of pair 4q's axis ("main") and of pair 4q + 3's axis ("second"; the same row except
// for q = 5, pairs 20..23 straddling frames/rows, and q = 10, pairs 40..43 straddling
// rows/columns). Both byte offsets move by lane constants per token and when the column (then
// the row) wraps. In a partial block the rows past the end repeat the last row and enter the
// sums multiplied by 0 (s + (+-0) = s, as s is never -0).
template <bool ROPE, bool FULL>
__device__ __forceinline__ void kstats_block(const PrepArgs& a, int j, int bh, int q) {
  const int r0 = j * BLK;
  const int valid = FULL ? BLK : min(BLK, a.N - r0);
  const uint16_t* Kh = a.K + ((size_t)bh * a.N + r0) * D + 8 * q;
  const char* ctab = reinterpret_cast<const char*>(a.rope_cos);
  const char* stab = reinterpret_cast<const char*>(a.rope_sin);
  int x = 0, y = 0;
  uint32_t om = 0, os = 0;                   // main / second table offsets (bytes)
  uint32_t sm = 0, ss = 0, xm = 0, xs = 0, ym = 0, ys = 0;  // their steps per token, x wrap, y wrap
  if (ROPE) {
    const int hw = a.Ht * a.Wd;
    const int f = r0 / hw, rem = r0 - f * hw;
    y = rem / a.Wd;
    x = rem - y * a.Wd;
    const int am = rope_axis(4 * q), as = rope_axis(4 * q + 3);
    auto offset = [&](int ax) { return (uint32_t)((ax == 0 ? f : (ax == 1 ? a.F + y : a.F + a.Ht + x)) * 256 + 16 * q); };
    auto step = [](int ax) { return ax == 2 ? 256u : 0u; };                                   // next column
    auto wrapx = [&](int ax) { return ax == 2 ? (uint32_t)(-256 * a.Wd) : (ax == 1 ? 256u : 0u); };  // next row
    auto wrapy = [&](int ax) { return ax == 1 ? (uint32_t)(-256 * a.Ht) : (ax == 0 ? 256u : 0u); };  // next frame
    om = offset(am);
    os = offset(as);
    sm = step(am);
    ss = step(as);
    xm = wrapx(am);
    xs = wrapx(as);
    ym = wrapy(am);
    ys = wrapy(as);
  }
  float s[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) s[c] = 0.f;
#pragma unroll 1
  for (int r = 0; r < BLK; r += 8) {
    u4 w[8];
    float4 cm[8], sn[8];
    float2 c2[8], s2[8];  // pairs 4q + 2, 4q + 3 from the second row
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int row = FULL ? r + u : min(r + u, valid - 1);
      w[u] = *reinterpret_cast<const u4*>(Kh + (uint32_t)row * 128u);
      if (ROPE) {
        cm[u] = *reinterpret_cast<const float4*>(ctab + om);
        sn[u] = *reinterpret_cast<const float4*>(stab + om);
        c2[u] = *reinterpret_cast<const float2*>(ctab + os + 8);
        s2[u] = *reinterpret_cast<const float2*>(stab + os + 8);
        if (FULL || r + u + 1 < valid) {
          om += sm;
          os += ss;
          if (++x == a.Wd) {
            x = 0;
            om += xm;
            os += xs;
            if (++y == a.Ht) {
              y = 0;
              om += ym;
              os += ys;
            }
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float v[8];
      unpack8(w[u], v);
      if (ROPE) {
        // pair 4q + 3 always from the second row, pair 4q + 2 from it only for q = 5
        const float cc[4] = {cm[u].x, cm[u].y, q == 5 ? c2[u].x : cm[u].z, c2[u].y};
        const float ssn[4] = {sn[u].x, sn[u].y, q == 5 ? s2[u].x : sn[u].z, s2[u].y};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float x0 = v[2 * k], x1 = v[2 * k + 1];
          const float pp = x1 * ssn[k], qq = x1 * cc[k];
          v[2 * k] = __builtin_fmaf(x0, cc[k], -pp);
          v[2 * k + 1] = __builtin_fmaf(x0, ssn[k], qq);
        }
      }
      if (!FULL) {
        const float keep = r + u < valid ? 1.f : 0.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) v[c] = v[c] * keep;
      }
#pragma unroll
      for (int c = 0; c < 8; ++c) s[c] = s[c] + v[c];
    }
  }
  float4* out = reinterpret_cast<float4*>(a.ws_ksum + ((size_t)bh * a.T + j) * D + 8 * q);
  out[0] = make_float4(s[0], s[1], s[2], s[3]);
  out[1] = make_float4(s[4], s[5], s[6], s[7]);
}

// Value statistics of block j: one pass over the gathered rows, keeping the sequential sum and
// the running maximum and minimum of each channel. With mu = bf16(sum / valid), the block's
// max |fl(x - mu)| is max(fl(xmax - mu), fl(mu - xmin)): fl(x - mu) is monotone in x and
// fl(mu - x) = -fl(x - mu). Lane q reads the row index of row r + q of each 16-row batch and
// the row's lanes broadcast it one row at a time. Rows past the end of a partial block repeat
// its last row (left out of the sums, no effect on the extrema).
template <bool FULL>
__device__ __forceinline__ void vstats_block(const PrepArgs& a, int j, int bh, int q) {
  const int r0 = j * BLK;
  const int valid = FULL ? BLK : min(BLK, a.N - r0);
  const size_t head = (size_t)bh * a.N;
  const uint16_t* Vh = a.V + head * D + 8 * q;
  const int32_t* ph = a.perm ? a.perm + head + r0 : nullptr;
  float s[8], hi[8], lo[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    s[c] = 0.f;
    hi[c] = -__builtin_inff();
    lo[c] = __builtin_inff();
  }
#pragma unroll 1
  for (int r = 0; r < BLK; r += 16) {
    const int row = FULL ? r + q : min(r + q, valid - 1);
    const int idx = ph ? clamp_index(ph[row], a.N) : r0 + row;
    u4 w[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int n = row_bcast_n(idx, u);
      w[u] = *reinterpret_cast<const u4*>(Vh + (uint32_t)n * 128u);
    }
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      float v[8];
      unpack8(w[u], v);
      const float keep = (FULL || r + u < valid) ? 1.f : 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        s[c] = s[c] + (FULL ? v[c] : v[c] * keep);
        hi[c] = fmaxf(hi[c], v[c]);
        lo[c] = fminf(lo[c], v[c]);
      }
    }
  }
  float mu[8];
  uint32_t mb[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint16_t b0 = 0, b1 = 0;
    if (a.smooth_v) {
      // full blocks divide by 128 (the same value as a multiply by 2^-7)
      b0 = f32_to_bf16(s[2 * k] / (float)valid);
      b1 = f32_to_bf16(s[2 * k + 1] / (float)valid);
    }
    mb[k] = (uint32_t)b0 | ((uint32_t)b1 << 16);
    mu[2 * k] = bf16_to_f32(b0);
    mu[2 * k + 1] = bf16_to_f32(b1);
  }
  *reinterpret_cast<u4*>(a.v_mean + ((size_t)bh * a.T + j) * D + 8 * q) = u4{mb[0], mb[1], mb[2], mb[3]};
  float m[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) m[c] = fmaxf(0.f, fmaxf(hi[c] - mu[c], mu[c] - lo[c]));
  float4* out = reinterpret_cast<float4*>(a.ws_vamax + ((size_t)bh * a.T + j) * D + 8 * q);
  out[0] = make_float4(m[0], m[1], m[2], m[3]);
  out[1] = make_float4(m[4], m[5], m[6], m[7]);
}

// grid (ceil(T/4), B*H, 1 + smooth_k), one wave: z = 0 value statistics, z = 1 key statistics
// of blocks 4 blockIdx.x .. + 3 (lanes 16g .. 16g + 15 take block 4 blockIdx.x + g).
template <bool ROPE>
__global__ __launch_bounds__(64) void prep_stats(PrepArgs a) {
  const int g = threadIdx.x >> 4, q = threadIdx.x & 15;
  const int j = 4 * blockIdx.x + g, bh = blockIdx.y;
  // the wave's blocks are all full unless the head's last block is among them and N % 128 != 0
  const bool full = (4 * blockIdx.x + 4) * BLK <= a.N;
  if (j >= a.T) return;
  if (blockIdx.z == 1) {
    if (full)
      kstats_block<ROPE, true>(a, j, bh, q);
    else
      kstats_block<ROPE, false>(a, j, bh, q);
  } else {
    if (full)
      vstats_block<true>(a, j, bh, q);
    else
      vstats_block<false>(a, j, bh, q);
  }
}

// ------------------------------------------------------------------------------------------
// Finalize, one workgroup per (head, 16-channel group): blockIdx.y < 8 forms the key channel
// mean of channels 16y .. 16y + 15 (sequential sum of the block sums in block order, one
// division by N); blockIdx.y >= 8 the per-channel residual scale amax/448 and 448/amax. The
// block partials are brought into LDS by the whole workgroup, up to FIN_CHUNK blocks at a time,
// so their loads are all in flight together.
// ------------------------------------------------------------------------------------------
constexpr int FIN_CHUNK = 512;

__global__ __launch_bounds__(256) void prep_finalize(PrepArgs a) {
  __shared__ float4 part[FIN_CHUNK][4];  // [block][4 channels x 4] of the group's 16 channels
  __shared__ float red[16][17];
  const int bh = blockIdx.x, t = threadIdx.x;
  const bool keys = blockIdx.y < 8;
  const int g = keys ? blockIdx.y : blockIdx.y - 8;
  const float* src = (keys ? a.ws_ksum : a.ws_vamax) + (size_t)bh * a.T * D + 16 * g;
  float acc = 0.f;  // keys: the running sum (threads 0..15); values: a partial max
  if (keys && !a.smooth_k) {
    if (t < 16) a.k_mean[(size_t)bh * D + 16 * g + t] = 0.f;
    return;
  }
  for (int j0 = 0; j0 < a.T; j0 += FIN_CHUNK) {
    const int nb = min(FIN_CHUNK, a.T - j0);
    __syncthreads();
    for (int e = t; e < nb * 4; e += 256)
      part[e >> 2][e & 3] = *reinterpret_cast<const float4*>(src + (size_t)(j0 + (e >> 2)) * D + 4 * (e & 3));
    __syncthreads();
    if (keys) {
      if (t < 16) {
        const float* col = reinterpret_cast<const float*>(part) + t;
        for (int jj = 0; jj < nb; ++jj) acc = acc + col[jj * 16];
      }
    } else {
      // channel t & 15, blocks (t >> 4), (t >> 4) + 16, ...
      const float* col = reinterpret_cast<const float*>(part) + (t & 15);
      for (int jj = t >> 4; jj < nb; jj += 16) acc = fmaxf(acc, col[jj * 16]);
    }
  }
  if (keys) {
    if (t < 16) a.k_mean[(size_t)bh * D + 16 * g + t] = acc / (float)a.N;
    return;
  }
  red[t >> 4][t & 15] = acc;
  __syncthreads();
  if (t < 16) {
    float amax = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) amax = fmaxf(amax, red[i][t]);
    const int c = 16 * g + t;
    a.v_scale[(size_t)bh * D + c] = amax > 0.f ? amax / 448.f : 1.f;
    a.ws_vinv[(size_t)bh * D + c] = amax > 0.f ? 448.f / amax : 0.f;
  }
}

// ------------------------------------------------------------------------------------------
// Quantization. A 128-row block per workgroup; 4 lanes per row, lane k4 = lane & 3 holding the
// 32 channels c = 32 i + 8 k4 + e (i, e = 0..3, 0..7): the loads are 16-byte row segments and
// the 128-point Walsh-Hadamard transform needs only two cross-lane stages (channel bits 3, 4).
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Cross-lane butterflies: every element becomes x + sgn * x_partner in one v_fmac_f32 whose
// first source is read from the partner lane of the quad (DPP quad_perm). The lower lane of a
// pair (sgn = +1) gets the sum of the butterfly; the upper lane (sgn = -1) gets
// x_upper - x_lower, the butterfly's difference with its sign flipped, and since
// fl(-d) = -fl(d) it is exactly that. The flipped sign is carried along and removed at the
// quantization. "s_nop 1" covers the wait states the hardware needs between a vector write and
// a DPP read of the same register.
#define VC_FMAC_DPP8(QP)                                                                                   \
  asm("s_nop 1\n\t"                                                                                      \
      "v_fmac_f32_dpp %0, %0, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %1, %1, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %2, %2, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %3, %3, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %4, %4, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %5, %5, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %6, %6, %8 " QP " row_mask:0xf bank_mask:0xf\n\t"                                 \
      "v_fmac_f32_dpp %7, %7, %8 " QP " row_mask:0xf bank_mask:0xf"                                     \
      : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7]) \
      : "v"(sgn))

__device__ __forceinline__ void cross_xor1(float (&v)[8], float sgn) { VC_FMAC_DPP8("quad_perm:[1,0,3,2]"); }
__device__ __forceinline__ void cross_xor2(float (&v)[8], float sgn) { VC_FMAC_DPP8("quad_perm:[2,3,0,1]"); }

// Butterfly stage h (channel bit b): lo <- lo + hi, hi <- lo - hi, in the order of the oracle.
// On return lane k4 holds sigma(k4) times the transform, sigma = (-1)^(bit0(k4) + bit1(k4)).
__device__ __forceinline__ void fwht_rows(float (&x)[4][8], int k4) {
  // bits 0..2: e, inside the lane
#pragma unroll
  for (int h = 1; h < 8; h <<= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if ((e & h) == 0) {
          const float lo = x[i][e], hi = x[i][e + h];
          x[i][e] = lo + hi;
          x[i][e + h] = lo - hi;
        }
  // bits 3, 4: k4, across lanes (xor 1, then xor 2; partners of the second stage carry the same
  // sign from the first, so it factors out)
  const float sg1 = (k4 & 1) ? -1.f : 1.f, sg2 = (k4 & 2) ? -1.f : 1.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) cross_xor1(x[i], sg1);
#pragma unroll
  for (int i = 0; i < 4; ++i) cross_xor2(x[i], sg2);
  // bits 5, 6: i, inside the lane
#pragma unroll
  for (int h = 1; h < 4; h <<= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if ((i & h) == 0)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float lo = x[i][e], hi = x[i + h][e];
          x[i][e] = lo + hi;
          x[i + h][e] = lo - hi;
        }
}

__device__ __forceinline__ void load_row32(const uint16_t* row, int k4, float (&x)[4][8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const u4 w = *reinterpret_cast<const u4*>(row + 32 * i + 8 * k4);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[i][2 * q] = bf16_lo(w[q]);
      x[i][2 * q + 1] = bf16_hi(w[q]);
    }
  }
}

// Rotary embedding of a lane's 32 channels (16 pairs 16 i + 4 k4 + 0..3) of token n.
__device__ __forceinline__ void rope_row32(float (&x)[4][8], int n, int k4, const PrepArgs& a) {
  const RopeRows rr = rope_rows(n, a);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // one 16-byte load per table from the row of the first pair's axis; the two quads that
    // cross an axis boundary (pairs 20..23 and 40..43) patch the pairs of the next axis
    const int p0 = 16 * i + 4 * k4;
    const int ax0 = rope_axis(p0);
    const int row = ax0 == 0 ? rr.f : (ax0 == 1 ? rr.y : rr.x);
    const uint32_t o = (uint32_t)(row * 64 + p0);
    float4 c4 = *reinterpret_cast<const float4*>(a.rope_cos + o);
    float4 s4 = *reinterpret_cast<const float4*>(a.rope_sin + o);
    if (i == 1 && k4 == 1) {
      const uint32_t oy = (uint32_t)(rr.y * 64);
      c4.z = a.rope_cos[oy + 22];
      c4.w = a.rope_cos[oy + 23];
      s4.z = a.rope_sin[oy + 22];
      s4.w = a.rope_sin[oy + 23];
    }
    if (i == 2 && k4 == 2) {
      const uint32_t ox = (uint32_t)(rr.x * 64);
      c4.w = a.rope_cos[ox + 43];
      s4.w = a.rope_sin[ox + 43];
    }
    const float cc[4] = {c4.x, c4.y, c4.z, c4.w}, ss[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
    for (int e = 0; e < 8; e += 2) {
      const float x0 = x[i][e], x1 = x[i][e + 1];
      const float pp = x1 * ss[e / 2], qq = x1 * cc[e / 2];
      x[i][e] = __builtin_fmaf(x0, cc[e / 2], -pp);
      x[i][e + 1] = __builtin_fmaf(x0, ss[e / 2], qq);
    }
  }
}

// Nearest E2M1 (MX FP4) code of v, |v| < 8: ties to the code with mantissa bit 0, saturating at
// 6, +0 for magnitudes that round to 0. With a = |v|, the code magnitude is rint(2a) below 2,
// 4 + rint(a - 2) on [2, 4) and 6 + rint((a - 4) / 2) on [4, 8) (each argument exact, so rint's
// ties to even are the format's ties), capped at 7.
__device__ __forceinline__ uint32_t fp4_code(float v) {
  const float a = fabsf(v);
  const float t = a < 2.f ? 2.f * a : (a < 4.f ? a - 2.f : __builtin_fmaf(a, 0.5f, -2.f));
  const float base = a < 2.f ? 0.f : (a < 4.f ? 4.f : 6.f);
  const uint32_t mag = (uint32_t)fminf(base + __builtin_rintf(t), 7.f);
  return mag | ((v < 0.f && mag != 0u) ? 8u : 0u);
}

// Q (IS_K = false) or K' (IS_K = true) rows of block j: gather, RoPE, centering (K), Hadamard,
// then, by the format QF: per-block symmetric INT8 (VC_QK_INT8: scale = amax/127, code =
// rint(x * (127/amax))), per-block symmetric E4M3 (VC_QK_FP8: scale = amax/448, code = the
// nearest-even E4M3 of x * (448/amax), +0 for codes of zero magnitude) or MXFP4 by 32-channel
// blocks (VC_QK_MXFP4: E8M0 scale byte floor(log2(amax)) - 2 + 127 per block).
template <bool IS_K, bool ROPE, bool HAD, int QF>
__device__ __forceinline__ void quant_qk(const PrepArgs& a, float* red, uint8_t* stage) {
  const int j = blockIdx.x, bh = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, k4 = lane & 3;
  const int r0 = j * BLK;
  const size_t head = (size_t)bh * a.N;
  const uint16_t* X = IS_K ? a.K : a.Q;
  const int32_t* gather = IS_K ? (a.perm ? a.perm + head : nullptr) : (a.q_perm ? a.q_perm + head : nullptr);

  float x[2][4][8];
  bool valid[2];
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int row = r0 + wave * 32 + it * 16 + (lane >> 2);
    valid[it] = row < a.N;
    const int n = valid[it] ? (gather ? clamp_index(gather[row], a.N) : row) : 0;
    load_row32(X + (head + n) * D, k4, x[it]);
    if (ROPE) rope_row32(x[it], n, k4, a);
    if (IS_K) {
      // the key mean (zeros without centering: x - 0 = x)
      const float* km = a.k_mean + (size_t)bh * D + 8 * k4;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float4 m0 = *reinterpret_cast<const float4*>(km + 32 * i);
        const float4 m1 = *reinterpret_cast<const float4*>(km + 32 * i + 4);
        const float mm[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) x[it][i][e] = x[it][i][e] - mm[e];
      }
    }
    if (HAD) fwht_rows(x[it], k4);
    if (!valid[it])
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) x[it][i][e] = 0.f;
  }

  const float sigma = HAD ? (((k4 ^ (k4 >> 1)) & 1) ? -1.f : 1.f) : 1.f;
  if constexpr (QF == VC_QK_MXFP4) {
    // channels 32 i .. 32 i + 31 of a row (one MX block) sit in the 4 lanes of the row's quad,
    // 8 each; lane (h*32 + r) of the scaled product's operand = row r, block 2m + h
    uint8_t* codes = reinterpret_cast<uint8_t*>(IS_K ? a.k : a.q) + ((size_t)bh * a.T + j) * (BLK * D / 2);
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int rl = wave * 32 + it * 16 + (lane >> 2), rb = rl >> 5, r = rl & 31;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float m = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(x[it][i][e]));
        m = fmaxf(m, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, m), 0xb1, 0xf, 0xf, true)));
        m = fmaxf(m, __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, m), 0x4e, 0xf, 0xf, true)));
        // floor(log2(m)) = exponent field - 127 for normal m; subnormal m clamps to byte 0
        const int ef = (int)((__float_as_uint(m) >> 23) & 0xffu);
        const int sb = m > 0.f ? max(ef - 2, 0) : 127;
        // sigma * 2^-X (exact scaling; the carried Hadamard sign restored)
        const float mult = sigma * __uint_as_float((uint32_t)(254 - sb) << 23);
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) w |= fp4_code(x[it][i][e] * mult) << (4 * e);
        const int mm = i >> 1, hh = i & 1;
        *reinterpret_cast<uint32_t*>(codes + ((rb * 2 + mm) * 2 + hh) * 512 + r * 16 + 4 * k4) = w;
        if (k4 == 0) stage[(hh * 32 + r) * 8 + rb * 2 + mm] = (uint8_t)sb;
      }
    }
    __syncthreads();
    if (threadIdx.x < 128)
      reinterpret_cast<uint32_t*>((IS_K ? a.k_mxs : a.q_mxs) + ((size_t)bh * a.T + j) * 512)[threadIdx.x] =
          reinterpret_cast<const uint32_t*>(stage)[threadIdx.x];
    return;
  }
  float m = 0.f;
#pragma unroll
  for (int it = 0; it < 2; ++it)
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(x[it][i][e]));
  m = wave_max(m);
  if (lane == 0) red[wave] = m;
  __syncthreads();
  const float amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  constexpr float top = QF == VC_QK_FP8 ? 448.f : 127.f;  // the largest code value
  const float inv = amax > 0.f ? top / amax : 0.f;
  if (threadIdx.x == 0) (IS_K ? a.k_scale : a.q_scale)[(size_t)bh * a.T + j] = amax > 0.f ? amax / top : 1.f;
  if constexpr (QF == VC_QK_FP8) {
    // x * (s inv) = s * fl(x inv) exactly, and E4M3 rounding is symmetric, so the carried
    // Hadamard sign goes into the multiplier; |fl(x inv)| <= 448 (1 + 2^-24)^2 converts to at most
    // 448. Lane k4 holds channels 8 k4 .. 8 k4 + 7 of each 32-channel block i = 2m + h: bytes
    // 8 (k4 & 1) .. of half k4 / 2 of the 32 bytes that lane (h*32 + r) of the FP8 product holds.
    const float mult = sigma * inv;
    uint8_t* codes = reinterpret_cast<uint8_t*>(IS_K ? a.k : a.q) + ((size_t)bh * a.T + j) * (BLK * D);
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int rl = wave * 32 + it * 16 + (lane >> 2), rb = rl >> 5, r = rl & 31;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t w[2];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const float* y = &x[it][i][4 * u];
          uint32_t v = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[0] * mult, y[1] * mult, 0, false);
          v = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[2] * mult, y[3] * mult, (int)v, true);
          // +0 for every code of zero magnitude (a zero's sign depends on the butterfly order)
          const uint32_t t = v & 0x7f7f7f7fu;
          w[u] = v & (((t + 0x7f7f7f7fu) & 0x80808080u) | 0x7f7f7f7fu);
        }
        const int off = ((((rb * 2 + (i >> 1)) * 2 + (i & 1)) * 2 + (k4 >> 1)) * 32 + r) * 16 + 8 * (k4 & 1);
        *reinterpret_cast<uint2*>(codes + off) = make_uint2(w[0], w[1]);
      }
    }
    return;
  }
  // the lane's sign from the cross-lane butterflies goes into the multiplier: x * (s inv) is
  // exactly s * fl(x inv). |fl(x inv)| <= 127 (1 + 2^-24)^2 < 127.5, so adding 1.5 * 2^23 rounds
  // it to the nearest integer, ties to even (the oracle's rint; its clamp to +-127 never acts),
  // and the low byte of the sum's bits is that integer in two's complement.
  const float mult = sigma * inv;
  int8_t* codes = (IS_K ? a.k : a.q) + ((size_t)bh * a.T + j) * (BLK * D);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int rl = wave * 32 + it * 16 + (lane >> 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t b[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) b[e] = __float_as_uint(x[it][i][e] * mult + 12582912.f);
      const uint32_t lo = __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u) | __builtin_amdgcn_perm(b[3], b[2], 0x04000c0cu);
      const uint32_t hi = __builtin_amdgcn_perm(b[5], b[4], 0x0c0c0400u) | __builtin_amdgcn_perm(b[7], b[6], 0x04000c0cu);
      *reinterpret_cast<uint2*>(codes + qk_tile_offset(rl, 32 * i + 8 * k4)) = make_uint2(lo, hi);
    }
  }
}

// V' rows of block j: gather, subtract the block mean (bf16; zeros without demeaning), scale per
// channel, E4M3 RNE, transposed through LDS into the tile order of the attention kernel.
__device__ __forceinline__ void quant_v(const PrepArgs& a, uint8_t (*vt)[D + 8]) {
  const int j = blockIdx.x, bh = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, k4 = lane & 3;
  const int r0 = j * BLK;
  const size_t head = (size_t)bh * a.N;
  const int32_t* gather = a.perm ? a.perm + head : nullptr;
  const uint16_t* mu = a.v_mean + ((size_t)bh * a.T + j) * D + 8 * k4;
  const float* vinv = a.ws_vinv + (size_t)bh * D + 8 * k4;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int rl = wave * 32 + it * 16 + (lane >> 2);
    const int row = r0 + rl;
    const bool valid = row < a.N;
    const int n = valid ? (gather ? clamp_index(gather[row], a.N) : row) : 0;
    float x[4][8];
    load_row32(a.V + (head + n) * D, k4, x);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const u4 mw = *reinterpret_cast<const u4*>(mu + 32 * i);
      const float4 i0 = *reinterpret_cast<const float4*>(vinv + 32 * i);
      const float4 i1 = *reinterpret_cast<const float4*>(vinv + 32 * i + 4);
      const float iv[8] = {i0.x, i0.y, i0.z, i0.w, i1.x, i1.y, i1.z, i1.w};
      uint32_t w2[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        // a channel whose residual is identically zero has vinv = 0: (+0) * 0 stores +0
        const float y0 = (x[i][e] - bf16_lo(mw[e / 2])) * iv[e];
        const float y1 = (x[i][e + 1] - bf16_hi(mw[e / 2])) * iv[e + 1];
        const uint32_t pk = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, 0, false) & 0xffffu;
        w2[e >> 2] |= pk << (16 * ((e >> 1) & 1));
      }
      if (!valid) w2[0] = w2[1] = 0u;
      *reinterpret_cast<uint2*>(&vt[rl][32 * i + 8 * k4]) = make_uint2(w2[0], w2[1]);
    }
  }
  __syncthreads();
  // transposed store: 1024 chunks of 16 bytes, 4 per thread; chunk = (kc, db, kh, sh, c)
  uint8_t* codes = a.v + ((size_t)bh * a.T + j) * (BLK * D);
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int chunk = threadIdx.x + 256 * u;
    const int c = chunk & 31, sh = (chunk >> 5) & 1, kh = (chunk >> 6) & 1, db = (chunk >> 7) & 3, kc = chunk >> 9;
    const int ch = 32 * db + c;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      const int key = 32 * (2 * kc + sh) + 8 * (t >> 2) + 4 * kh + (t & 3);
      w[t >> 2] |= (uint32_t)vt[key][ch] << (8 * (t & 3));
    }
    *reinterpret_cast<u4*>(codes + (size_t)chunk * 16) = u4{w[0], w[1], w[2], w[3]};
  }
}

// grid (T, B*H, 3): z = 0 K' rows, z = 1 V' rows, z = 2 Q rows of block blockIdx.x.
template <bool ROPE, bool HAD, int QF>
__global__ __launch_bounds__(256) void prep_quant(PrepArgs a) {
  __shared__ float red[4];
  // V codes of the block, row-major (8-byte rows), for the transpose; MX scale bytes of a Q/K block
  __shared__ uint8_t vt[BLK][D + 8];
  // K' and V' first: their rows were just read by the statistics pass and may still be cached
  if (blockIdx.z == 0)
    quant_qk<true, ROPE, HAD, QF>(a, red, &vt[0][0]);
  else if (blockIdx.z == 1)
    quant_v(a, vt);
  else
    quant_qk<false, ROPE, HAD, QF>(a, red, &vt[0][0]);
}

hipError_t launch_prep(const PrepArgs& a, int BH, hipStream_t s) {
  const dim3 sgrid((a.T + 3) / 4, BH, a.smooth_k ? 2 : 1);
  if (a.rope)
    prep_stats<true><<<sgrid, 64, 0, s>>>(a);
  else
    prep_stats<false><<<sgrid, 64, 0, s>>>(a);
  prep_finalize<<<dim3(BH, 16), 256, 0, s>>>(a);
  const dim3 grid(a.T, BH, 3);
  auto quant = [&](auto QFC) {
    constexpr int qf = decltype(QFC)::value;
    if (a.rope) {
      if (a.hadamard)
        prep_quant<true, true, qf><<<grid, 256, 0, s>>>(a);
      else
        prep_quant<true, false, qf><<<grid, 256, 0, s>>>(a);
    } else {
      if (a.hadamard)
        prep_quant<false, true, qf><<<grid, 256, 0, s>>>(a);
      else
        prep_quant<false, false, qf><<<grid, 256, 0, s>>>(a);
    }
  };
  if (a.qk_fmt == VC_QK_MXFP4)
    quant(std::integral_constant<int, VC_QK_MXFP4>{});
  else if (a.qk_fmt == VC_QK_FP8)
    quant(std::integral_constant<int, VC_QK_FP8>{});
  else
    quant(std::integral_constant<int, VC_QK_INT8>{});
  return hipGetLastError();
}

}  // namespace vc
