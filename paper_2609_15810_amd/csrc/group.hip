// Value-guided grouping (Sec. 3.2 "Value-guided permutation"): per (batch, head) the value tokens
// are clustered and the keys/values are later gathered in cluster order.
//
// KMEANS: Lloyd rounds on per-head INT8 codes of V (scale amax/127 over the head).
//   grp_amax     per-head max |V|, one partial maximum per 256 tokens (max is order-free)
//   grp_codes    the head's maximum from the partials, INT8 codes, row-major [N][128]
//   grp_init     initial integer centroids (tokens floor((2c+1)N/(2k)), or the caller's fp32
//                centroids requantized)
//   grp_assign   1024 tokens per workgroup in chunks of 256, on the matrix cores: the INT8
//                product C X^T gives |C|^2 - 2 x.C exactly in int32, the argmin is one integer
//                min over (distance << 7 | cluster) (ties to the smallest cluster); then the
//                exact member sums O X with the one-hot label matrix O as the INT8 A operand
//                (the chunk's codes transposed through LDS), and the counts (partials per
//                workgroup, reduced by grp_update)
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

// Each workgroup reduces 64 KB of the head (16 chunks of 16 bytes per thread, all loads issued
// before the first use; chunks past the head's end re-read its last chunk) to one partial maximum.
__global__ __launch_bounds__(256) void grp_amax(GroupArgs a) {
  __shared__ float red[4];
  const int bh = blockIdx.y;
  const size_t words = (size_t)a.N * D / 8;  // 16-byte chunks of the head
  const u4* src = reinterpret_cast<const u4*>(a.V + (size_t)bh * a.N * D);
  u4 w[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) w[u] = src[min(((size_t)blockIdx.x * 16 + u) * 256 + threadIdx.x, words - 1)];
  float m = 0.f;
#pragma unroll
  for (int u = 0; u < 16; ++u)
#pragma unroll
    for (int q = 0; q < 4; ++q) m = fmaxf(m, fmaxf(fabsf(bf16_lo(w[u][q])), fabsf(bf16_hi(w[u][q]))));
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0)   // one partial per workgroup (gridDim.x = nblk), reduced by grp_codes
    reinterpret_cast<float*>(a.counts)[(size_t)bh * gridDim.x + blockIdx.x] =
        fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__device__ __forceinline__ float head_amax(const GroupArgs& a, int bh) { return a.scale[bh]; }

// 256 tokens per workgroup: consecutive threads quantize consecutive 16-byte chunks of the
// workgroup's rows (8 channels each) and store the 8 code bytes, so loads and stores coalesce.
__global__ __launch_bounds__(256) void grp_codes(GroupArgs a) {
  __shared__ float red[4];
  const int bh = blockIdx.y, t = threadIdx.x;
  const int n0 = blockIdx.x * 256;
  const int ntok = min(256, a.N - n0);
  // the head's |V| maximum from grp_amax's partials (one per 256-token block; max is order-free)
  float pm = 0.f;
  for (int i = t; i < (int)gridDim.x; i += 256) pm = fmaxf(pm, reinterpret_cast<const float*>(a.counts)[(size_t)bh * gridDim.x + i]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) pm = fmaxf(pm, __shfl_xor(pm, o));
  if ((t & 63) == 0) red[t >> 6] = pm;
  __syncthreads();
  const float amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  if (blockIdx.x == 0 && t == 0) a.scale[bh] = amax;   // for the centroid kernels
  const float inv = amax > 0.f ? 127.f / amax : 0.f;
  const u4* src = reinterpret_cast<const u4*>(a.V + ((size_t)bh * a.N + n0) * D);
  uint2* dst = reinterpret_cast<uint2*>(a.codes + ((size_t)bh * a.N + n0) * D);
  u4 w[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) w[u] = src[min(u * 256 + t, ntok * 16 - 1)];   // chunks of padded tokens re-read the last one
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int q = u * 256 + t;
    if ((q >> 4) >= ntok) continue;
    uint32_t pk[2] = {0u, 0u};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float f = (e & 1) ? bf16_hi(w[u][e >> 1]) : bf16_lo(w[u][e >> 1]);
      float r = __builtin_rintf(f * inv);
      r = fminf(fmaxf(r, -127.f), 127.f);
      pk[e >> 2] |= ((uint32_t)((int)r & 0xff)) << (8 * (e & 3));
    }
    dst[q] = make_uint2(pk[0], pk[1]);
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

constexpr int AW = 8;            // waves per assignment workgroup
constexpr int ATOK = 1024;       // tokens per assignment workgroup (one partial each)
constexpr int ACH = 256;         // tokens per chunk: one 32-token label step per wave
constexpr int NCH = ATOK / ACH;

// One Lloyd assignment on the matrix cores (KB = clusters / 32, rounded up), chunk by chunk.
// Labels (wave w: tokens 32w .. 32w + 31 of the chunk):
//   S^T = C X^T     INT8 MFMA 32x32x32, A = centroid rows (registers), B = the tokens' codes;
//                   lane (token l%32, half l/32) holds 16 clusters' x.C, the other 16 in lane l^32
//   key  = (|C|^2 - 2 x.C + 2^23) << 7 | cluster, argmin = integer min of the keys (the distance
//          fits 24 bits, the cluster 7 bits; equal distances resolve to the smaller cluster)
//   the label goes to memory, to the chunk's label row in LDS and to its cluster's count; the
//   codes go to the chunk's LDS rows.
// Sums (wave w: byte w%4 of every 4-channel word, i.e. channels 4c + w%4, half w/4 of the chunk):
//   sums += O X     INT8 MFMA, A = one-hot labels (cluster rows x 32 tokens), B = 16 consecutive
//                   tokens of channel 4 col + w%4 per lane, gathered from the LDS rows
// Each wave keeps 16 sum registers per cluster block. The sums are added into LDS and written as
// one partial per workgroup; all arithmetic is integer, so the order of additions is free.
template <int KB>
__global__ __launch_bounds__(AW * 64) void grp_assign(GroupArgs a) {
  __shared__ int32_t acc[KB * 32][D];
  __shared__ int32_t cntl[KB * 32];
  __shared__ int32_t norm[KB * 32];
  __shared__ __attribute__((aligned(16))) uint8_t lab[ACH];
  __shared__ __attribute__((aligned(16))) uint32_t xs[ACH][D / 4 + 2];   // 136-byte rows: no bank conflicts
  const int bh = blockIdx.y, wg = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kh = lane >> 5, col = lane & 31, K = a.k, N = a.N;
  for (int i = tid; i < KB * 32 * D; i += AW * 64) (&acc[0][0])[i] = 0;
  if (tid < KB * 32) {
    norm[tid] = a.cnorm[(size_t)bh * KMAX + tid];
    cntl[tid] = 0;
  }
  const int8_t* codes = a.codes + (size_t)bh * N * D;
  const int wbase = wg * ATOK;
  // centroid rows as the A operand (padding clusters are zero rows) and the lane's norms
  v4i ca[KB][4];
  int32_t nr[KB][16];
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int dc = 0; dc < 4; ++dc)
      ca[cb][dc] = *reinterpret_cast<const v4i*>(a.cent8 + ((size_t)bh * KMAX + 32 * cb + col) * D + 32 * dc + 16 * kh);
  // the lane's codes (token 32 wave + col of a chunk, channels 32 dc + 16 kh ..), one chunk ahead
  auto load_codes = [&](int c, v4i (&x)[4]) __attribute__((always_inline)) {
    const int8_t* xr = codes + (size_t)min(wbase + c * ACH + 32 * wave + col, N - 1) * D + 16 * kh;
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) x[dc] = *reinterpret_cast<const v4i*>(xr + 32 * dc);
  };
  v4i xb[4];
  load_codes(0, xb);
  __syncthreads();
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) nr[cb][r] = norm[32 * cb + 8 * (r >> 2) + 4 * kh + (r & 3)];
  const int db = wave & 3, half = wave >> 2;
  // byte db of each of two words -> bytes 0, 1 (lo) or 2, 3 (hi) of the result
  const uint32_t sel_lo = 0x0c0c0000u | ((uint32_t)(4 + db) << 8) | (uint32_t)db;
  const uint32_t sel_hi = ((uint32_t)(4 + db) << 24) | ((uint32_t)db << 16) | 0x0c0cu;
  v16i sums[KB];
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) sums[cb][r] = 0;

  for (int c = 0; c < NCH; ++c) {
    const int cbase = wbase + c * ACH;
    if (cbase >= N) break;   // uniform over the workgroup
    {
      const int n0 = cbase + 32 * wave;
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
      if (kh == 0) {
        lab[32 * wave + col] = (uint8_t)label;
        if (valid) {
          a.labels[(size_t)bh * N + token] = label;
          atomicAdd(&cntl[label], 1);
        }
      }
      // codes into the chunk's LDS rows (tokens past N: zero codes); rows are 136 bytes, so the
      // stores are 8-byte ones
#pragma unroll
      for (int dc = 0; dc < 4; ++dc) {
        const v4i v = valid ? xb[dc] : v4i{0, 0, 0, 0};
        uint2* d = reinterpret_cast<uint2*>(&xs[32 * wave + col][8 * dc + 4 * kh]);
        d[0] = make_uint2((uint32_t)v[0], (uint32_t)v[1]);
        d[1] = make_uint2((uint32_t)v[2], (uint32_t)v[3]);
      }
      if (c + 1 < NCH) load_codes(c + 1, xb);   // the next chunk's codes in flight
    }
    __syncthreads();
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
      const int t0 = 128 * half + 32 * s4;   // step's first token in the chunk
      if (cbase + t0 >= N) break;
      // operand: tokens t0 + 16 kh .. + 15 of channel 4 col + db, byte i = token i
      int32_t xv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r0 = t0 + 16 * kh + 4 * q;
        const uint32_t lo = __builtin_amdgcn_perm(xs[r0 + 1][col], xs[r0][col], sel_lo);
        const uint32_t hi = __builtin_amdgcn_perm(xs[r0 + 3][col], xs[r0 + 2][col], sel_hi);
        xv[q] = (int32_t)(lo | hi);
      }
      const v4i xop = {xv[0], xv[1], xv[2], xv[3]};
      const u4 l4 = *reinterpret_cast<const u4*>(&lab[t0 + 16 * kh]);
#pragma unroll
      for (int cb = 0; cb < KB; ++cb) {
        const uint32_t rep = (uint32_t)(32 * cb + col) * 0x01010101u;
        int32_t oh[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t x = l4[q] ^ rep;
          const uint32_t nz = (((x & 0x7f7f7f7fu) + 0x7f7f7f7fu) | x) & 0x80808080u;   // 0x80 where byte != 0
          oh[q] = (int32_t)((~nz >> 7) & 0x01010101u);
        }
        const v4i ohv = {oh[0], oh[1], oh[2], oh[3]};
        sums[cb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(ohv, xop, sums[cb], 0, 0, 0);
      }
    }
    __syncthreads();   // the next chunk overwrites the rows and labels
  }
  // this wave's sums (rows = clusters, column col = channel 4 col + db) into the LDS accumulators
#pragma unroll
  for (int cb = 0; cb < KB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 32 * cb + 8 * (r >> 2) + 4 * kh + (r & 3);
      if (row < K) atomicAdd(&acc[row][4 * col + db], sums[cb][r]);
    }
  __syncthreads();
  const size_t part = (size_t)bh * a.npart + wg;
  for (int i = tid; i < K * D; i += AW * 64) a.sums[part * K * D + i] = (&acc[0][0])[i];
  if (tid < K) a.counts[part * K + tid] = cntl[tid];
}

// per-256-token-block label counts of the final labels (the stable sort's histogram), stored
// label-major [lab][blk]
__global__ __launch_bounds__(GT) void grp_hist(GroupArgs a) {
  __shared__ int32_t h[KMAX];
  const int blk = blockIdx.x, bh = blockIdx.y, t = threadIdx.x;
  if (t < KMAX) h[t] = 0;
  __syncthreads();
  const int n = blk * GT + t;
  if (n < a.N) atomicAdd(&h[a.labels[(size_t)bh * a.N + n]], 1);
  __syncthreads();
  if (t < a.nlab) a.counts[((size_t)bh * a.nlab + t) * a.nblk + blk] = h[t];
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

// label-major exclusive offsets of the per-block label counts: off[k][b]. Each thread sums a
// contiguous run of the label-major counts, a scan over the 256 run sums, then each thread writes
// its run's offsets.
__global__ __launch_bounds__(256) void grp_offsets(GroupArgs a) {
  __shared__ int32_t part[256];
  const int bh = blockIdx.x, t = threadIdx.x;
  const int total = a.nlab * a.nblk;
  const int per = (total + 255) / 256;
  const int lo = min(total, t * per), hi = min(total, lo + per);
  const int32_t* cnt = a.counts + (size_t)bh * a.nblk * a.nlab;   // [lab][blk]
  int32_t s = 0;
  for (int idx = lo; idx < hi; ++idx) s += cnt[idx];
  part[t] = s;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {   // inclusive scan (integers: exact in any order)
    const int32_t v = t >= o ? part[t - o] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int32_t run = part[t] - s;
  int32_t* off = a.blockhist + (size_t)bh * a.nlab * a.nblk;   // [lab][blk]
  for (int idx = lo; idx < hi; ++idx) {
    off[idx] = run;
    run += cnt[idx];
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
  // grp_amax's grid (16 chunks of 16 bytes per thread = 256 tokens per workgroup) equals grp_codes'
  grp_amax<<<tok, 256, 0, s>>>(a);
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
