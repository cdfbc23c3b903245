// Value-guided grouping (Sec. 3.2 "Value-guided permutation"): per (batch, head) the value tokens
// are clustered and the keys/values are later gathered in cluster order.
//
// KMEANS: Lloyd rounds on per-head INT8 codes of V (scale amax/127 over the head).
//   grp_amax     per-head max |V| (exact, order-free: integer max of non-negative float bits)
//   grp_codes    INT8 codes, row-major [N][128], plus a token-interleaved copy for the member
//                sums (per 32-token block, per 32-channel block and lane half: 16 consecutive
//                tokens of one channel; transposed through LDS)
//   grp_init     initial integer centroids (tokens floor((2c+1)N/(2k)), or the caller's fp32
//                centroids requantized)
//   grp_assign   1024 tokens per workgroup, 32 per wave step, on the matrix cores: the INT8
//                product C X^T gives |C|^2 - 2 x.C exactly in int32, the argmin is one integer
//                min over (distance << 7 | cluster) (ties to the smallest cluster); then the
//                exact member sums O X with the one-hot label matrix O as the INT8 A operand,
//                and the counts (partials per workgroup, reduced by grp_update)
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

// 256 tokens per workgroup: each thread quantizes one token into its row-major row and into LDS;
// then 4x4 byte transposes through LDS write the token-interleaved copy with 16-byte stores.
__global__ __launch_bounds__(256) void grp_codes(GroupArgs a) {
  __shared__ __attribute__((aligned(16))) uint32_t xs[256][D / 4 + 1];
  const int bh = blockIdx.y, t = threadIdx.x;
  const int n = blockIdx.x * 256 + t;
  const float amax = head_amax(a, bh);
  const float inv = amax > 0.f ? 127.f / amax : 0.f;
  if (n < a.N) {
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
        xs[t][4 * ch + q] = pk;
      }
      dst[ch] = u4{out[0], out[1], out[2], out[3]};
    }
  } else {
#pragma unroll
    for (int w = 0; w < D / 4; ++w) xs[t][w] = 0u;   // padded tokens: zero codes
  }
  __syncthreads();
  // unit (block b of 32 tokens, lane half kh, channels 4g..4g+3): 16 tokens x 4 channels
  const int ntb = (a.N + 31) / 32;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int unit = u * 256 + t;
    const int g = unit & 31, kh = (unit >> 5) & 1, b = unit >> 6;
    const int tb = blockIdx.x * 8 + b;
    if (tb >= ntb) continue;
    uint32_t col[4][4];   // col[j][tq]: channel 4g+j of tokens 4tq..4tq+3 (of the 16)
#pragma unroll
    for (int tq = 0; tq < 4; ++tq) {
      uint32_t r[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) r[e] = xs[b * 32 + kh * 16 + 4 * tq + e][g];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        col[j][tq] = ((r[0] >> (8 * j)) & 0xffu) | (((r[1] >> (8 * j)) & 0xffu) << 8) |
                     (((r[2] >> (8 * j)) & 0xffu) << 16) | (((r[3] >> (8 * j)) & 0xffu) << 24);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = 4 * g + j, db = c >> 5, cl = c & 31;
      u4* dst = reinterpret_cast<u4*>(a.codesT + ((size_t)bh * ntb + tb) * (32 * D) + (((db * 2 + kh) * 32 + cl) * 16));
      *dst = u4{col[j][0], col[j][1], col[j][2], col[j][3]};
    }
  }
}

constexpr int NORM_PAD = 8388000;    // |C|^2 of a padding cluster: above every real distance

// Centroid k of head bh is kept three ways: int32 (the exact state of the Lloyd rounds), int8
// (the assignment's A operand; the values are means of int8 codes, so they fit) and its squared
// norm. Rows k..KMAX-1 are padding: zero codes, norm NORM_PAD. One thread per channel.
__device__ __forceinline__ void publish_centroid(const GroupArgs& a, int bh, int k, int c, int32_t v) {
  __shared__ int32_t red[D / 64];
  a.cent[((size_t)bh * a.k + k) * D + c] = v;
  a.cent8[((size_t)bh * KMAX + k) * D + c] = (int8_t)v;
  int32_t sq = v * v;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) sq += __shfl_xor(sq, o);
  if ((c & 63) == 0) red[c >> 6] = sq;
  __syncthreads();
  if (c == 0) a.cnorm[(size_t)bh * KMAX + k] = red[0] + red[1];
}

__global__ __launch_bounds__(D) void grp_init(GroupArgs a) {
  const int k = blockIdx.x, bh = blockIdx.y, c = threadIdx.x;
  if (k >= a.k) {   // padding rows
    a.cent8[((size_t)bh * KMAX + k) * D + c] = 0;
    if (c == 0) a.cnorm[(size_t)bh * KMAX + k] = NORM_PAD;
    return;
  }
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
  publish_centroid(a, bh, k, c, v);
}

constexpr int AW = 4;            // waves per assignment workgroup
constexpr int AG = 8;            // 32-token steps per wave
constexpr int ATOK = AW * AG * 32;   // 1024 tokens per assignment workgroup

// One Lloyd assignment on the matrix cores (KB = clusters / 32, rounded up). Per 32-token step:
//   S^T = C X^T     INT8 MFMA 32x32x32, A = centroid rows (registers), B = the tokens' codes;
//                   lane (token l%32, half l/32) holds 16 clusters' x.C, the other 16 in lane l^32
//   key  = (|C|^2 - 2 x.C + 2^23) << 7 | cluster, argmin = integer min of the keys (the distance
//          fits 24 bits, the cluster 7 bits; equal distances resolve to the smaller cluster)
//   sums += O X     INT8 MFMA, A = one-hot labels (cluster rows x 32 tokens), B = the
//                   token-interleaved codes (16 consecutive tokens of one channel per lane)
//   counts         popcounts of the one-hot bytes
// The wave's sums stay in registers; at the end they are added into LDS and written as one
// partial per workgroup.
template <int KB>
__global__ __launch_bounds__(AW * 64) void grp_assign(GroupArgs a) {
  __shared__ int32_t acc[KB * 32][D];
  __shared__ int32_t cntl[KB * 32];
  __shared__ int32_t norm[KB * 32];
  __shared__ __attribute__((aligned(16))) uint8_t lab[AW][32];
  const int bh = blockIdx.y, wg = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kh = lane >> 5, col = lane & 31, K = a.k, N = a.N;
  for (int i = tid; i < KB * 32 * D; i += AW * 64) (&acc[0][0])[i] = 0;
  if (tid < KB * 32) {
    norm[tid] = a.cnorm[(size_t)bh * KMAX + tid];
    cntl[tid] = 0;
  }
  // centroid rows as the A operand (padding clusters are zero rows) and the lane's norms
  v4i ca[KB][4];
  int32_t nr[KB][16];
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int dc = 0; dc < 4; ++dc)
      ca[cb][dc] = *reinterpret_cast<const v4i*>(a.cent8 + ((size_t)bh * KMAX + 32 * cb + col) * D + 32 * dc + 16 * kh);
  __syncthreads();
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) nr[cb][r] = norm[32 * cb + 8 * (r >> 2) + 4 * kh + (r & 3)];

  const int ntb = (N + 31) / 32;
  const int8_t* codes = a.codes + (size_t)bh * N * D;
  const int8_t* codesT = a.codesT + (size_t)bh * ntb * (32 * D);
  v16i sums[KB][4];
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) sums[cb][db][r] = 0;
  int32_t cntp[KB];
#pragma unroll
  for (int cb = 0; cb < KB; ++cb) cntp[cb] = 0;

  auto load_step = [&](int n0, v4i (&xb)[4], v4i (&xt)[4]) {
    const int token = min(n0 + col, N - 1);
    const int8_t* xr = codes + (size_t)token * D + 16 * kh;
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) xb[dc] = *reinterpret_cast<const v4i*>(xr + 32 * dc);
    const int8_t* xc = codesT + (size_t)(n0 >> 5) * (32 * D) + (kh * 32 + col) * 16;
#pragma unroll
    for (int db = 0; db < 4; ++db) xt[db] = *reinterpret_cast<const v4i*>(xc + db * 1024);
  };
  const int nbase = wg * ATOK + wave * (AG * 32);
  v4i xb[4], xt[4];
  if (nbase < N) load_step(nbase, xb, xt);
  for (int g = 0; g < AG; ++g) {
    const int n0 = nbase + g * 32;
    if (n0 >= N) break;
    v4i xbn[4], xtn[4];
    if (g + 1 < AG && n0 + 32 < N) load_step(n0 + 32, xbn, xtn);   // next step's codes in flight
    int best = 0x7fffffff;
#pragma unroll
    for (int cb = 0; cb < KB; ++cb) {
      v16i S = {};
#pragma unroll
      for (int dc = 0; dc < 4; ++dc) S = __builtin_amdgcn_mfma_i32_32x32x32_i8(ca[cb][dc], xb[dc], S, 0, 0, 0);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = ((nr[cb][r] - 2 * S[r] + (1 << 23)) << 7) | (32 * cb + 8 * (r >> 2) + 4 * kh + (r & 3));
        best = min(best, key);
      }
    }
    best = min(best, __shfl_xor(best, 32));
    const int token = n0 + col;
    const bool valid = token < N;
    const int label = valid ? (best & 127) : 255;
    if (valid && kh == 0) a.labels[(size_t)bh * N + token] = label;
    if (kh == 0) lab[wave][col] = (uint8_t)label;
    // the wave's 32 labels: one-hot bytes of (cluster row, token) for this lane's 16 tokens
    const u4 l4 = *reinterpret_cast<const u4*>(&lab[wave][16 * kh]);
#pragma unroll
    for (int cb = 0; cb < KB; ++cb) {
      const uint32_t rep = (uint32_t)(32 * cb + col) * 0x01010101u;
      int32_t oh[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t x = l4[q] ^ rep;
        const uint32_t nz = (((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x) & 0x80808080u;   // 0x80 where byte != 0
        oh[q] = (int32_t)((~nz >> 7) & 0x01010101u);
        cntp[cb] += __builtin_popcount((uint32_t)oh[q]);
      }
      const v4i ohv = {oh[0], oh[1], oh[2], oh[3]};
#pragma unroll
      for (int db = 0; db < 4; ++db) sums[cb][db] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ohv, xt[db], sums[cb][db], 0, 0, 0);
    }
    if (g + 1 < AG && n0 + 32 < N) {
#pragma unroll
      for (int q = 0; q < 4; ++q) { xb[q] = xbn[q]; xt[q] = xtn[q]; }
    }
  }
  // this wave's sums and counts into the workgroup's LDS accumulators
#pragma unroll
  for (int cb = 0; cb < KB; ++cb) {
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * cb + 8 * (r >> 2) + 4 * kh + (r & 3);
        if (row < K) atomicAdd(&acc[row][32 * db + col], sums[cb][db][r]);
      }
    if (32 * cb + col < K) atomicAdd(&cntl[32 * cb + col], cntp[cb]);
  }
  __syncthreads();
  const size_t part = (size_t)bh * a.npart + wg;
  for (int i = tid; i < K * D; i += AW * 64) a.sums[part * K * D + i] = (&acc[0][0])[i];
  if (tid < K) a.counts[part * K + tid] = cntl[tid];
}

// per-256-token-block label counts of the final labels (the stable sort's histogram)
__global__ __launch_bounds__(GT) void grp_hist(GroupArgs a) {
  __shared__ int32_t h[KMAX];
  const int blk = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
  if (t < KMAX) h[t] = 0;
  __syncthreads();
  const int n = blk * GT + t;
  if (n < a.N) atomicAdd(&h[a.labels[(size_t)bh * a.N + n]], 1);
  __syncthreads();
  if (t < a.nlab) a.counts[((size_t)bh * a.nblk + blk) * a.nlab + t] = h[t];
}

__device__ __forceinline__ int32_t div_rne(long long num, long long den) {
  long long q = num / den, rem = num % den;
  if (rem < 0) { q -= 1; rem += den; }
  if (2 * rem > den || (2 * rem == den && (q & 1))) q += 1;
  return (int32_t)q;
}

__global__ __launch_bounds__(D) void grp_update(GroupArgs a) {
  const int k = blockIdx.x, bh = blockIdx.y, c = threadIdx.x;
  long long S = 0, cnt = 0;
  for (int b0 = 0; b0 < a.npart; b0 += 32) {   // integer sums: any order; loads issued 32 ahead
    int32_t sv[32], cv[32];
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const size_t p = ((size_t)bh * a.npart + min(b0 + u, a.npart - 1)) * a.k + k;
      sv[u] = a.sums[p * D + c];
      cv[u] = a.counts[p];
    }
#pragma unroll
    for (int u = 0; u < 32; ++u)
      if (b0 + u < a.npart) { S += sv[u]; cnt += cv[u]; }
  }
  if (cnt > 0) publish_centroid(a, bh, k, c, div_rne(S, cnt));   // an empty cluster keeps its centroid
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
  grp_init<<<dim3(KMAX, BH), D, 0, s>>>(a);
  const int rounds = a.iters > 0 ? a.iters : 1;
  for (int it = 0; it < rounds; ++it) {
    if (a.k <= 32) grp_assign<1><<<dim3(a.npart, BH), AW * 64, 0, s>>>(a);
    else grp_assign<2><<<dim3(a.npart, BH), AW * 64, 0, s>>>(a);
    if (a.iters > 0) grp_update<<<dim3(a.k, BH), 128, 0, s>>>(a);
  }
  grp_cent_out<<<dim3(a.k, BH), 128, 0, s>>>(a);
  grp_hist<<<dim3(a.nblk, BH), GT, 0, s>>>(a);
  grp_offsets<<<BH, 256, 0, s>>>(a);
  grp_scatter<<<dim3(a.nblk, BH), GT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace vc
