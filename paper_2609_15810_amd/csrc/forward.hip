// 8-bit VC-Attention forward on gfx950 matrix cores (Sec. 3.1 eq. tiled-low-bit-attention,
// Sec. 3.2 eq. vc-online-update, Sec. 3.3 eq. direct-fp8).
//
// One workgroup = one 128-row query block of one (batch, head); four waves of 32 queries, one wave
// per SIMD. Both products are computed transposed so that a lane owns one query:
//   S^T = K_hat Q_hat^T   INT8 MFMA 32x32x32 (A = key rows from LDS, B = the wave's queries held
//                         in registers for the whole kernel);
//   O^T += V_hat^T P^T    FP8 MFMA 32x32x64 (A = residual codes from LDS, B = P codes).
// A lane's 16 results of a 32-key block are 16 keys of its own query, so the running row maximum
// is an in-register max plus one exchange with lane l^32, alpha and l are per-lane scalars, and the
// ExpCast-FP8 codes (one fp32 fma and one round-to-nearest-even byte conversion per score) are
// already in the B-operand order of the FP8 product: byte s of lane half kh in key chunk kc is key
// 32(2kc + s/16) + 8((s%16)/4) + 4kh + s%4, the order in which the preprocessing stores V_hat.
//
// Throughput measures (the kernel is bound by the vector ALU work between the two products):
//   - the probability row sum r comes from the matrix cores: an all-ones E4M3 A operand times the
//     P codes;
//   - the block mean is restored in batches of 8 tiles: r_j (rescaled with A) is kept per lane and
//     every 8 tiles O^T += M^T R is one bf16 matrix product with mu_j / s_V and r split into
//     hi + lo bf16 parts (hi*hi + hi*lo + lo*hi, relative error ~2^-16);
//   - the rescale of A by alpha is skipped when no row maximum of the wave moved;
//   - software pipelining: while the vector units turn tile j's scores into codes, the matrix
//     cores run the scores of tile j+1 and the value product of tile j-1.
// The code of every score is the one-rounding fma(float(acc), 8a, fl(fl(120 + beta) - 8m')) of the
// method's fp32 formula, clipped by the saturating byte conversion (round to nearest even).
// K_hat (one tile ahead) and V_hat (one tile behind) are double-buffered in LDS and fetched through
// registers one iteration before use. Tiles are visited in ascending order with the running
// maximum updated once per 128-key tile, the schedule on which the codes are defined.
#include "vc_common.hpp"
#include "vc_internal.hpp"

namespace vc {

constexpr int FWD_THREADS = 256;
constexpr int TILE_BYTES = BLK * D;  // 16384

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

struct FwdSmem {
  uint8_t k[2][TILE_BYTES];
  uint8_t v[2][TILE_BYTES];
  uint16_t u[2][2][D][8];  // [chunk parity][hi, lo][channel][tile slot]: mu_j / s_V as bf16 hi + lo
  float sv[D];
};

__device__ __forceinline__ v16i mfma_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mfma_f8(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// S^T of one 128-key tile for the wave's 32 queries (exact int32).
__device__ __forceinline__ void qk_tile(const uint8_t* kt, const v4i (&qop)[4], int kh, int col, v16i (&s)[4]) {
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
    for (int r = 0; r < 16; ++r) s[kb][r] = 0;
#pragma unroll
    for (int dc = 0; dc < 4; ++dc) {
      const v4i kop = *reinterpret_cast<const v4i*>(kt + ((kb * 4 + dc) * 2 + kh) * 512 + col * 16);
      s[kb] = mfma_i8(kop, qop[dc], s[kb]);
    }
  }
}

// O^T += V_hat^T P^T of one tile.
__device__ __forceinline__ void pv_tile(const uint8_t* vt, const v8i (&pop)[2], int kh, int col, v16f (&o)[4]) {
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const int base = ((((kc * 4 + db) * 2 + kh) * 2) * 32 + col) * 16;
      const u4 lo = *reinterpret_cast<const u4*>(vt + base);
      const u4 hi = *reinterpret_cast<const u4*>(vt + base + 512);
      const v8i vop = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
      o[db] = mfma_f8(vop, pop[kc], o[db]);
    }
}

// Running maximum and probability codes of one tile. Padded keys of the last tile hold INT_MIN
// (excluded from the maximum; their codes are cleared by clear_padded). Returns alpha, updates m_run.
template <int PMODE>
__device__ __forceinline__ void softmax_tile(const v16i (&s)[4], float a_s, float cbias, float& m_run, float& alpha,
                                             v8i (&pop)[2]) {
  int mx = INT_MIN;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 16; r += 2) mx = max(mx, max(s[kb][r], s[kb][r + 1]));
  mx = max(mx, __shfl_xor(mx, 32));
  const float m_new = fmaxf(m_run, (float)mx * a_s);
  alpha = __builtin_amdgcn_exp2f(m_run - m_new);
  m_run = m_new;
  if (PMODE == 0) {
    const float a8 = 8.f * a_s;
    const float bias = cbias - 8.f * m_new;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int d4 = 0; d4 < 4; ++d4) {
          uint32_t w = 0;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            w = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_fmaf((float)s[2 * kc + half][4 * d4 + q], a8, bias), q, w);
          pop[kc][4 * half + d4] = (int)w;
        }
  } else {
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int d4 = 0; d4 < 4; ++d4) {
          float p[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float t = (float)s[2 * kc + half][4 * d4 + q] * a_s;
            p[q] = __builtin_amdgcn_exp2f(t - m_new) * 256.f;
          }
          uint32_t w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], 0, false);
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], (int)w, true);
          pop[kc][4 * half + d4] = (int)w;
        }
  }
}

// Padded keys of the last tile (key >= kvalid): INT_MIN scores before the softmax ...
__device__ __forceinline__ void mask_tile(v16i (&s)[4], int kh, int kvalid) {
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (32 * kb + 8 * (r >> 2) + 4 * kh + (r & 3) >= kvalid) s[kb][r] = INT_MIN;
}

// ... and zero probability codes after it.
__device__ __forceinline__ void clear_padded(v8i (&pop)[2], int kh, int kvalid) {
#pragma unroll
  for (int kc = 0; kc < 2; ++kc)
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      uint32_t keep = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int key = 32 * (2 * kc + (w >> 2)) + 8 * (w & 3) + 4 * kh + q;
        if (key < kvalid) keep |= 0xffu << (8 * q);
      }
      pop[kc][w] = (int)((uint32_t)pop[kc][w] & keep);
    }
}

__device__ __forceinline__ uint16_t bf16_bits(float f) { return f32_to_bf16(f); }

template <int PMODE>
__global__ __launch_bounds__(FWD_THREADS, 1) void attn_fwd(FwdArgs a) {
  __shared__ __attribute__((aligned(16))) FwdSmem sm;
  const int qt = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kh = lane >> 5, col = lane & 31;
  const int T = a.T;
  const size_t tile0 = (size_t)bh * T;

  // the wave's 32 queries as the B operand of the score product (4 chunks of 32 channels)
  const int8_t* qblk = a.q + (tile0 + qt) * TILE_BYTES;
  v4i qop[4];
#pragma unroll
  for (int dc = 0; dc < 4; ++dc) qop[dc] = *reinterpret_cast<const v4i*>(qblk + ((wave * 4 + dc) * 2 + kh) * 512 + col * 16);
  const float sq = a.q_scale[tile0 + qt];

  float inv_sv = 0.f;
  if (tid < D) {
    const float s = a.v_scale[(size_t)bh * D + tid];
    sm.sv[tid] = s;
    inv_sv = 1.f / s;
  }

  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + tile0 * TILE_BYTES;
  const uint8_t* vbase = a.v + tile0 * TILE_BYTES;
  u4 kst[4], vst[4];
  float mu_st = 0.f;
  auto fetch_k = [&](int j) {  // K_hat tile j and its block mean (tile index clamped to T-1)
    j = min(j, T - 1);
#pragma unroll
    for (int u = 0; u < 4; ++u) kst[u] = *reinterpret_cast<const u4*>(kbase + (size_t)j * TILE_BYTES + u * 4096 + tid * 16);
    mu_st = (a.smooth_v && tid < D) ? bf16_to_f32(a.v_mean[(tile0 + j) * D + tid]) * inv_sv : 0.f;
  };
  auto fetch_v = [&](int j) {
#pragma unroll
    for (int u = 0; u < 4; ++u) vst[u] = *reinterpret_cast<const u4*>(vbase + (size_t)j * TILE_BYTES + u * 4096 + tid * 16);
  };
  auto stash_k = [&](int buf, int tile) {
#pragma unroll
    for (int u = 0; u < 4; ++u) *reinterpret_cast<u4*>(&sm.k[buf][u * 4096 + tid * 16]) = kst[u];
    if (tid < D) {
      const uint16_t hi = bf16_bits(mu_st);
      const uint16_t lo = bf16_bits(mu_st - bf16_to_f32(hi));
      sm.u[(tile >> 3) & 1][0][tid][tile & 7] = hi;
      sm.u[(tile >> 3) & 1][1][tid][tile & 7] = lo;
    }
  };
  auto stash_v = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) *reinterpret_cast<u4*>(&sm.v[buf][u * 4096 + tid * 16]) = vst[u];
  };

  // prologue: K_0, K_1 (and their means) in LDS, the V buffer read by the empty first value product
  // zeroed, S of tile 0 computed
  fetch_k(0);
  stash_k(0, 0);
  fetch_k(1);
  stash_k(1, 1);
#pragma unroll
  for (int u = 0; u < 4; ++u) *reinterpret_cast<u4*>(&sm.v[1][u * 4096 + tid * 16]) = u4{0u, 0u, 0u, 0u};
  __syncthreads();

  v16i sa[4], sb[4];
  qk_tile(sm.k[0], qop, kh, col, sa);
  if (T == 1) mask_tile(sa, kh, a.N);

  v16f o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  v8i pa[2], pb[2];
#pragma unroll
  for (int w = 0; w < 8; ++w) { pa[0][w] = 0; pa[1][w] = 0; pb[0][w] = 0; pb[1][w] = 0; }
  float R[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) R[t] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const v8i ones = {0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838};

  // flush the batched block means of chunk `par`: O^T += M^T R (bf16 hi/lo products)
  auto flush_means = [&](int par) {
    bf16x8 b;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint16_t hi = bf16_bits(R[t]);
      const uint16_t v = kh == 0 ? hi : bf16_bits(R[t] - bf16_to_f32(hi));
      b[t] = __builtin_bit_cast(__bf16, v);
    }
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      const int c = 32 * db + col;
      const bf16x8 a_hi = *reinterpret_cast<const bf16x8*>(&sm.u[par][0][c][0]);
      bf16x8 a_lo = *reinterpret_cast<const bf16x8*>(&sm.u[par][1][c][0]);
      if (kh) a_lo = bf16x8{};
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_hi, b, o[db], 0, 0, 0);
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_lo, b, o[db], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) R[t] = 0.f;
  };

  // one pipeline step: tile j's softmax while the matrix cores do S of tile j+1 and PV of tile j-1
  auto step = [&](int j, v16i (&s_cur)[4], v16i (&s_nxt)[4], v8i (&p_cur)[2], v8i (&p_prev)[2]) {
    fetch_k(j + 2);
    fetch_v(j);
    const float a_s = (sq * a.k_scale[tile0 + j]) * a.kappa;
    float alpha;
    qk_tile(sm.k[(j + 1) & 1], qop, kh, col, s_nxt);
    pv_tile(sm.v[(j + 1) & 1], p_prev, kh, col, o);
    softmax_tile<PMODE>(s_cur, a_s, a.cbias, m_run, alpha, p_cur);
    if (j == T - 1) clear_padded(p_cur, kh, a.N - (T - 1) * BLK);
    v16f rs = {};
    rs = mfma_f8(ones, p_cur[0], rs);
    rs = mfma_f8(ones, p_cur[1], rs);
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
#pragma unroll
      for (int t = 0; t < 8; ++t) R[t] *= alpha;
    }
    const float r = rs[0];
    l_run = alpha * l_run + r;
    const int slot = j & 7;
#pragma unroll
    for (int t = 0; t < 8; ++t) R[t] = t == slot ? r : R[t];
    if (a.smooth_v && slot == 7) flush_means((j >> 3) & 1);
    stash_k(j & 1, j + 2);
    stash_v(j & 1);
    if (j == T - 2) mask_tile(s_nxt, kh, a.N - (T - 1) * BLK);
    __syncthreads();
  };

  int j = 0;
  for (; j + 1 < T; j += 2) {
    step(j, sa, sb, pa, pb);
    step(j + 1, sb, sa, pb, pa);
  }
  if (j < T) {
    step(j, sa, sb, pa, pb);
    pv_tile(sm.v[j & 1], pa, kh, col, o);      // value product of the last tile (P in pa)
  } else {
    pv_tile(sm.v[(j - 1) & 1], pb, kh, col, o);  // last tile was j-1, its P in pb
  }
  if (a.smooth_v && (T & 7) != 0) flush_means(((T - 1) >> 3) & 1);

  // epilogue: O = A s_V / l, bf16, row q written to token q_perm[q] (or q)
  const int q = qt * BLK + wave * 32 + col;
  if (q < a.N) {
    const float inv_l = 1.f / l_run;
    const int qo = a.q_perm ? clamp_index(a.q_perm[(size_t)bh * a.N + q], a.N) : q;
    uint16_t* orow = a.O + ((size_t)bh * a.N + qo) * D;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c0 = 32 * db + 8 * g + 4 * kh;
        const uint32_t w0 = (uint32_t)f32_to_bf16(o[db][4 * g + 0] * sm.sv[c0 + 0] * inv_l) |
                            ((uint32_t)f32_to_bf16(o[db][4 * g + 1] * sm.sv[c0 + 1] * inv_l) << 16);
        const uint32_t w1 = (uint32_t)f32_to_bf16(o[db][4 * g + 2] * sm.sv[c0 + 2] * inv_l) |
                            ((uint32_t)f32_to_bf16(o[db][4 * g + 3] * sm.sv[c0 + 3] * inv_l) << 16);
        *reinterpret_cast<uint2*>(orow + c0) = make_uint2(w0, w1);
      }
  }
}

hipError_t launch_forward(const FwdArgs& a, int BH, hipStream_t s) {
  const dim3 grid(a.T, BH);
  if (a.p_mode == 0) attn_fwd<0><<<grid, FWD_THREADS, 0, s>>>(a);
  else attn_fwd<1><<<grid, FWD_THREADS, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace vc
