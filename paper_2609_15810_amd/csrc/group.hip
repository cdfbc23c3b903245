// Value-guided grouping (Sec. 3.2 "Value-guided permutation"): per (batch, head) the value tokens
// are clustered and the keys/values are later gathered in cluster order.
//
// KMEANS: Lloyd rounds on per-head INT8 codes of V (scale amax/127 over the head).
//   grp_amax     per-head max |V| (exact, order-free: integer max of non-negative float bits)
//   grp_codes    INT8 codes, row-major [N][128]
//   grp_init     initial integer centroids (tokens floor((2c+1)N/(2k)), or the caller's fp32
//                centroids requantized)
//   grp_assign   256 tokens per workgroup: squared-L2 argmin |C|^2 - 2 x.C in int32 with
//                v_dot4 (ties to the smallest cluster), then exact integer member sums and
//                counts of the workgroup's tokens (partials, reduced by grp_update)
//   grp_update   centroid = round-half-even integer mean of the members (exact int64 division)
// Integer arithmetic throughout makes labels, centroids and the permutation reproducible bit for
// bit regardless of the order in which partial sums are combined.
// Sort: per-block label counts -> label-major exclusive offsets -> stable scatter (rank among
// equal labels by token index), i.e. a stable counting sort: perm lists tokens by label, then
// by index.
// CUBE: static cube order in closed form; IDENTITY: perm = 0..N-1.
#include "vc_common.hpp"
#include "vc_internal.hpp"

namespace vc {

constexpr int GT = 256;   // tokens per assignment / sort block
constexpr int KMAX = 64;  // clusters supported by the kernels

__global__ void grp_zero(uint32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// Each workgroup reduces 64 KB of the head (16 chunks of 16 bytes per thread) before one atomic.
__global__ __launch_bounds__(256) void grp_amax(GroupArgs a) {
  __shared__ float red[4];
  const int bh = blockIdx.y;
  const size_t words = (size_t)a.N * D / 8;  // 16-byte chunks of the head
  const u4* src = reinterpret_cast<const u4*>(a.V + (size_t)bh * a.N * D);
  float m = 0.f;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const size_t i = ((size_t)blockIdx.x * 16 + u) * 256 + threadIdx.x;
    if (i < words) {
      const u4 w = src[i];
#pragma unroll
      for (int q = 0; q < 4; ++q) m = fmaxf(m, fmaxf(fabsf(bf16_lo(w[q])), fabsf(bf16_hi(w[q]))));
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0)
    atomicMax(reinterpret_cast<unsigned int*>(a.scale) + bh,
              __float_as_uint(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))));
}

__device__ __forceinline__ float head_amax(const GroupArgs& a, int bh) { return a.scale[bh]; }

__global__ __launch_bounds__(256) void grp_codes(GroupArgs a) {
  const int bh = blockIdx.y;
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= a.N) return;
  const float amax = head_amax(a, bh);
  const float inv = amax > 0.f ? 127.f / amax : 0.f;
  const u4* src = reinterpret_cast<const u4*>(a.V + ((size_t)bh * a.N + n) * D);
  u4* dst = reinterpret_cast<u4*>(a.codes + ((size_t)bh * a.N + n) * D);
#pragma unroll
  for (int ch = 0; ch < 8; ++ch) {   // 16 channels per chunk
    const u4 w0 = src[2 * ch], w1 = src[2 * ch + 1];
    uint32_t out[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t w = q < 2 ? w0[2 * q] : w1[2 * (q - 2)];
      const uint32_t v = q < 2 ? w0[2 * q + 1] : w1[2 * (q - 2) + 1];
      float f[4] = {bf16_lo(w), bf16_hi(w), bf16_lo(v), bf16_hi(v)};
      uint32_t pk = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float r = __builtin_rintf(f[e] * inv);
        r = fminf(fmaxf(r, -127.f), 127.f);
        pk |= ((uint32_t)((int)r & 0xff)) << (8 * e);
      }
      out[q] = pk;
    }
    dst[ch] = u4{out[0], out[1], out[2], out[3]};
  }
}

__global__ __launch_bounds__(128) void grp_init(GroupArgs a) {
  const int k = blockIdx.x, bh = blockIdx.y, c = threadIdx.x;
  int32_t v;
  if (a.warm_start) {
    const float amax = head_amax(a, bh);
    const float inv = amax > 0.f ? 127.f / amax : 0.f;
    float r = __builtin_rintf(a.centroids[((size_t)bh * a.k + k) * D + c] * inv);
    r = fminf(fmaxf(r, -127.f), 127.f);
    v = (int32_t)r;
  } else {
    const long long n0 = ((long long)(2 * k + 1) * a.N) / (2LL * a.k);
    v = a.codes[((size_t)bh * a.N + n0) * D + c];
  }
  a.cent[((size_t)bh * a.k + k) * D + c] = v;
}

__global__ __launch_bounds__(GT) void grp_assign(GroupArgs a) {
  __shared__ int32_t cent8[KMAX][D / 4];   // centroids as packed int8 words
  __shared__ int32_t norm[KMAX];
  __shared__ uint8_t xs[GT][D + 4];
  __shared__ int32_t lab[GT];
  __shared__ int32_t acc[2][KMAX][D];
  const int blk = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
  const int K = a.k;
  const int32_t* C = a.cent + (size_t)bh * K * D;
  for (int idx = t; idx < K * (D / 4); idx += GT) {
    const int k = idx / (D / 4), w = idx % (D / 4);
    const int32_t* c4 = C + (size_t)k * D + 4 * w;
    cent8[k][w] = (c4[0] & 0xff) | ((c4[1] & 0xff) << 8) | ((c4[2] & 0xff) << 16) | ((c4[3] & 0xff) << 24);
  }
  for (int idx = t; idx < 2 * KMAX * D; idx += GT) (&acc[0][0][0])[idx] = 0;
  if (t < K) {
    int32_t s = 0;
    for (int c = 0; c < D; ++c) s += C[(size_t)t * D + c] * C[(size_t)t * D + c];
    norm[t] = s;
  }
  __syncthreads();

  const int n = blk * GT + t;
  const bool valid = n < a.N;
  int32_t xw[D / 4];
  const u4* src = reinterpret_cast<const u4*>(a.codes + ((size_t)bh * a.N + (valid ? n : 0)) * D);
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const u4 w = src[q];
    xw[4 * q] = (int32_t)w[0]; xw[4 * q + 1] = (int32_t)w[1]; xw[4 * q + 2] = (int32_t)w[2]; xw[4 * q + 3] = (int32_t)w[3];
  }
  int best = 0;
  int32_t bd = 0;
  for (int k = 0; k < K; ++k) {
    int32_t dot = 0;
#pragma unroll
    for (int w = 0; w < D / 4; ++w) dot = __builtin_amdgcn_sdot4(xw[w], cent8[k][w], dot, false);
    const int32_t dist = norm[k] - 2 * dot;
    if (k == 0 || dist < bd) { bd = dist; best = k; }
  }
  lab[t] = valid ? best : -1;
  if (valid) a.labels[(size_t)bh * a.N + n] = best;
#pragma unroll
  for (int w = 0; w < D / 4; ++w) *reinterpret_cast<int32_t*>(&xs[t][4 * w]) = xw[w];
  __syncthreads();

  // exact member sums of this block: thread (half, c) walks its 128 tokens
  {
    const int c = t & (D - 1), half = t >> 7;
    for (int i = 0; i < GT / 2; ++i) {
      const int tok = half * (GT / 2) + i;
      const int L = lab[tok];
      if (L >= 0) acc[half][L][c] += (int32_t)(int8_t)xs[tok][c];
    }
  }
  __syncthreads();
  const size_t pbase = ((size_t)bh * a.nblk + blk) * K;
  for (int idx = t; idx < K * D; idx += GT) {
    const int k = idx / D, c = idx % D;
    a.sums[(pbase + k) * D + c] = acc[0][k][c] + acc[1][k][c];
  }
  if (t < K) {
    int32_t cnt = 0;
    for (int i = 0; i < GT; ++i) cnt += (lab[i] == t);
    a.counts[pbase + t] = cnt;
  }
}

__device__ __forceinline__ int32_t div_rne(long long num, long long den) {
  long long q = num / den, rem = num % den;
  if (rem < 0) { q -= 1; rem += den; }
  if (2 * rem > den || (2 * rem == den && (q & 1))) q += 1;
  return (int32_t)q;
}

__global__ __launch_bounds__(128) void grp_update(GroupArgs a) {
  const int k = blockIdx.x, bh = blockIdx.y, c = threadIdx.x;
  long long S = 0, cnt = 0;
  for (int b0 = 0; b0 < a.nblk; b0 += 16) {   // integer sums: any order; loads issued 16 ahead
    int32_t sv[16], cv[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const size_t p = ((size_t)bh * a.nblk + min(b0 + u, a.nblk - 1)) * a.k + k;
      sv[u] = a.sums[p * D + c];
      cv[u] = a.counts[p];
    }
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (b0 + u < a.nblk) { S += sv[u]; cnt += cv[u]; }
  }
  if (cnt > 0) a.cent[((size_t)bh * a.k + k) * D + c] = div_rne(S, cnt);
}

__global__ __launch_bounds__(128) void grp_cent_out(GroupArgs a) {
  const int k = blockIdx.x, bh = blockIdx.y, c = threadIdx.x;
  const float amax = head_amax(a, bh);
  const float scale = amax > 0.f ? amax / 127.f : 1.f;
  const size_t i = ((size_t)bh * a.k + k) * D + c;
  a.centroids[i] = (float)a.cent[i] * scale;
}

// label-major exclusive offsets of the per-block label counts: off[k][b]
__global__ __launch_bounds__(256) void grp_offsets(GroupArgs a) {
  __shared__ int32_t part[256];
  const int bh = blockIdx.x, t = threadIdx.x;
  const int total = a.nlab * a.nblk;
  const int per = (total + 255) / 256;
  const int lo = min(total, t * per), hi = min(total, lo + per);
  const int32_t* cnt = a.counts + (size_t)bh * a.nblk * a.nlab;   // [blk][lab]
  int32_t s = 0;
  for (int idx = lo; idx < hi; ++idx) s += cnt[(size_t)(idx % a.nblk) * a.nlab + idx / a.nblk];
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int32_t run = 0;
    for (int i = 0; i < 256; ++i) { const int32_t v = part[i]; part[i] = run; run += v; }
  }
  __syncthreads();
  int32_t run = part[t];
  int32_t* off = a.blockhist + (size_t)bh * a.nlab * a.nblk;   // [lab][blk]
  for (int idx = lo; idx < hi; ++idx) {
    off[idx] = run;
    run += cnt[(size_t)(idx % a.nblk) * a.nlab + idx / a.nblk];
  }
}

__global__ __launch_bounds__(GT) void grp_scatter(GroupArgs a) {
  __shared__ int32_t lab[GT];
  const int blk = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
  const int n = blk * GT + t;
  lab[t] = n < a.N ? a.labels[(size_t)bh * a.N + n] : -1;
  __syncthreads();
  if (n >= a.N) return;
  const int L = lab[t];
  int rank = 0;
  for (int i = 0; i < t; ++i) rank += (lab[i] == L);
  const int pos = a.blockhist[((size_t)bh * a.nlab + L) * a.nblk + blk] + rank;
  a.perm[(size_t)bh * a.N + pos] = n;
  if (a.inv_perm) a.inv_perm[(size_t)bh * a.N + n] = pos;
}

// Static cube order in closed form: the tokens of all cubes before cube (ca, cb, cc) in raster
// order, plus the token's raster rank inside its (possibly clipped) cube.
__global__ __launch_bounds__(256) void grp_cube(GroupArgs a) {
  const int bh = blockIdx.y;
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= a.N) return;
  const int x = n % a.Wd, y = (n / a.Wd) % a.Ht, f = n / (a.Wd * a.Ht);
  const int ca = f / a.cube_t, cb = y / a.cube_h, cc = x / a.cube_w;
  const int ft = min(a.cube_t, a.F - ca * a.cube_t), ht = min(a.cube_h, a.Ht - cb * a.cube_h);
  const int wt = min(a.cube_w, a.Wd - cc * a.cube_w);
  const long long pos = (long long)ca * a.cube_t * a.Ht * a.Wd +
                        (long long)ft * ((long long)cb * a.cube_h * a.Wd + (long long)ht * cc * a.cube_w) +
                        (long long)(f - ca * a.cube_t) * ht * wt + (long long)(y - cb * a.cube_h) * wt + (x - cc * a.cube_w);
  const int ny = (a.Ht + a.cube_h - 1) / a.cube_h, nx = (a.Wd + a.cube_w - 1) / a.cube_w;
  a.labels[(size_t)bh * a.N + n] = (ca * ny + cb) * nx + cc;
  a.perm[(size_t)bh * a.N + pos] = n;
  if (a.inv_perm) a.inv_perm[(size_t)bh * a.N + n] = (int32_t)pos;
}

__global__ __launch_bounds__(256) void grp_identity(GroupArgs a) {
  const int bh = blockIdx.y;
  const int n = blockIdx.x * 256 + threadIdx.x;
  if (n >= a.N) return;
  a.labels[(size_t)bh * a.N + n] = 0;
  a.perm[(size_t)bh * a.N + n] = n;
  if (a.inv_perm) a.inv_perm[(size_t)bh * a.N + n] = n;
}

hipError_t launch_group(const GroupArgs& a, int BH, hipStream_t s) {
  const dim3 tok((a.N + 255) / 256, BH);
  if (a.mode == 0) {
    grp_identity<<<tok, 256, 0, s>>>(a);
    return hipGetLastError();
  }
  if (a.mode == 1) {
    grp_cube<<<tok, 256, 0, s>>>(a);
    return hipGetLastError();
  }
  grp_zero<<<(BH + 255) / 256, 256, 0, s>>>(reinterpret_cast<uint32_t*>(a.scale), BH);
  const size_t words = (size_t)a.N * D / 8;
  grp_amax<<<dim3((unsigned)((words + 4095) / 4096), BH), 256, 0, s>>>(a);
  grp_codes<<<tok, 256, 0, s>>>(a);
  grp_init<<<dim3(a.k, BH), 128, 0, s>>>(a);
  const int rounds = a.iters > 0 ? a.iters : 1;
  for (int it = 0; it < rounds; ++it) {
    grp_assign<<<dim3(a.nblk, BH), GT, 0, s>>>(a);
    if (a.iters > 0) grp_update<<<dim3(a.k, BH), 128, 0, s>>>(a);
  }
  grp_cent_out<<<dim3(a.k, BH), 128, 0, s>>>(a);
  grp_offsets<<<BH, 256, 0, s>>>(a);
  grp_scatter<<<dim3(a.nblk, BH), GT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace vc
