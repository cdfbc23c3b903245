// 8-bit VC-Attention forward on gfx950 matrix cores (Sec. 3.1 eq. tiled-low-bit-attention,
// Sec. 3.2 eq. vc-online-update, Sec. 3.3 eq. direct-fp8).
//
// One workgroup = one 128-row query block of one (batch, head), four waves of 32 queries.
// Both products are computed transposed so that a lane owns one query:
//   S^T = K_hat Q_hat^T   INT8 MFMA 32x32x32 (A = key rows from LDS, B = the wave's queries
//                         held in registers for the whole kernel), int32 accumulators;
//   O^T += V_hat^T P^T    FP8 MFMA 32x32x64 (A = residual codes from LDS, B = P codes).
// A lane's 16 int32 results of one 32-key block hold 16 keys of its own query, so
//   - the running row maximum is an in-register max plus one exchange with lane l^32,
//   - the probability codes written by ExpCast-FP8 (one fp32 fma and one round-to-nearest-even
//     byte conversion per score) are already laid out as the B operand of the FP8 product:
//     byte s of lane half kh in key chunk kc stands for key 32(2kc + s/16) + 8((s%16)/4)
//     + 4kh + s%4, and the residual codes are stored in exactly that key order by the
//     preprocessing,
//   - alpha, l and the probability row sum r are per-lane scalars.
// The block mean is restored as A <- alpha A + r mu_j / s_V before the FP8 product adds P R_hat,
// and the epilogue writes O = A s_V / l in bf16.
// K_hat and V_hat tiles (16 KB each) are double-buffered in LDS; the next tile is fetched into
// registers while the current one is consumed. Tiles are visited in ascending order and the
// running maximum is updated once per 128-key tile, the schedule the codes are defined on.
#include "vc_common.hpp"
#include "vc_internal.hpp"

namespace vc {

constexpr int FWD_WAVES = 4;
constexpr int FWD_THREADS = 64 * FWD_WAVES;
constexpr int TILE_BYTES = BLK * D;  // 16384

struct FwdSmem {
  uint8_t k[2][TILE_BYTES];
  uint8_t v[2][TILE_BYTES];
  float mu[2][D];  // mu_j / s_V of the tile (code units of the residual)
  float sv[D];
};

__device__ __forceinline__ v16i mfma_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mfma_f8(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// Probability codes of one 128-key tile into the two FP8 B operands (keys 0..63, 64..127).
// MASK: the last tile, where keys >= kvalid are padding and get P = 0.
template <int PMODE, bool MASK>
__device__ __forceinline__ void encode_p(const v16i (&s)[4], float a_s, float m_new, float cbias, int kh,
                                         int kvalid, v8i (&pop)[2]) {
  const float a8 = 8.f * a_s;
  const float bias = cbias - 8.f * m_new;
#pragma unroll
  for (int kc = 0; kc < 2; ++kc)
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int kb = 2 * kc + half;
#pragma unroll
      for (int d4 = 0; d4 < 4; ++d4) {
        uint32_t w = 0;
        if (PMODE == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int r = 4 * d4 + q;
            float f = __builtin_fmaf((float)s[kb][r], a8, bias);
            if (MASK && 32 * kb + 8 * d4 + 4 * kh + q >= kvalid) f = -1.f;
            w = __builtin_amdgcn_cvt_pk_u8_f32(f, q, w);
          }
        } else {
          float p[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int r = 4 * d4 + q;
            const float t = (float)s[kb][r] * a_s;
            p[q] = __builtin_amdgcn_exp2f(t - m_new) * 256.f;
            if (MASK && 32 * kb + 8 * d4 + 4 * kh + q >= kvalid) p[q] = 0.f;
          }
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(p[0], p[1], 0, false);
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(p[2], p[3], (int)w, true);
        }
        pop[kc][4 * half + d4] = (int)w;
      }
    }
}

template <int PMODE>
__global__ __launch_bounds__(FWD_THREADS) void attn_fwd(FwdArgs a) {
  __shared__ __attribute__((aligned(16))) FwdSmem sm;
  const int qt = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kh = lane >> 5, col = lane & 31;
  const size_t tile0 = (size_t)bh * a.T;

  // this wave's 32 queries as the B operand of the score product (4 chunks of 32 channels)
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
  u4 stg[8];
  float mu_stg = 0.f;
  auto fetch = [&](int j) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      stg[u] = *reinterpret_cast<const u4*>(kbase + (size_t)j * TILE_BYTES + u * 4096 + tid * 16);
      stg[4 + u] = *reinterpret_cast<const u4*>(vbase + (size_t)j * TILE_BYTES + u * 4096 + tid * 16);
    }
    if (a.smooth_v && tid < D) mu_stg = bf16_to_f32(a.v_mean[(tile0 + j) * D + tid]) * inv_sv;
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      *reinterpret_cast<u4*>(&sm.k[buf][u * 4096 + tid * 16]) = stg[u];
      *reinterpret_cast<u4*>(&sm.v[buf][u * 4096 + tid * 16]) = stg[4 + u];
    }
    if (tid < D) sm.mu[buf][tid] = mu_stg;
  };

  fetch(0);
  stash(0);
  __syncthreads();

  float m_run = -INFINITY, l_run = 0.f;
  v16f o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;

  for (int j = 0; j < a.T; ++j) {
    const int buf = j & 1;
    if (j + 1 < a.T) fetch(j + 1);
    const float a_s = (sq * a.k_scale[tile0 + j]) * a.kappa;

    // S^T = K_hat Q_hat^T (exact int32)
    v16i s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0;
#pragma unroll
      for (int dc = 0; dc < 4; ++dc) {
        const v4i kop = *reinterpret_cast<const v4i*>(&sm.k[buf][((kb * 4 + dc) * 2 + kh) * 512 + col * 16]);
        s[kb] = mfma_i8(kop, qop[dc], s[kb]);
      }
    }

    // running maximum over the tile's valid keys (int32, then one scale)
    const bool last = (j == a.T - 1);
    const int kvalid = a.N - j * BLK;
    int mx = INT_MIN;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * kb + 8 * (r >> 2) + 4 * kh + (r & 3);
        const int v = (last && key >= kvalid) ? INT_MIN : s[kb][r];
        mx = max(mx, v);
      }
    mx = max(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, (float)mx * a_s);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);

    v8i pop[2];
    if (last) encode_p<PMODE, true>(s, a_s, m_new, a.cbias, kh, kvalid, pop);
    else encode_p<PMODE, false>(s, a_s, m_new, a.cbias, kh, kvalid, pop);

    // probability row sum of the decoded codes (exact in fp32)
    float rs = 0.f;
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        const v2f lo = __builtin_amdgcn_cvt_pk_f32_fp8(pop[kc][w], false);
        const v2f hi = __builtin_amdgcn_cvt_pk_f32_fp8(pop[kc][w], true);
        rs += (lo[0] + lo[1]) + (hi[0] + hi[1]);
      }
    rs += __shfl_xor(rs, 32);

    // A <- alpha A + r mu_j / s_V
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    if (a.smooth_v) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const float4 mu = *reinterpret_cast<const float4*>(&sm.mu[buf][32 * db + 8 * g + 4 * kh]);
          o[db][4 * g + 0] = __builtin_fmaf(rs, mu.x, o[db][4 * g + 0]);
          o[db][4 * g + 1] = __builtin_fmaf(rs, mu.y, o[db][4 * g + 1]);
          o[db][4 * g + 2] = __builtin_fmaf(rs, mu.z, o[db][4 * g + 2]);
          o[db][4 * g + 3] = __builtin_fmaf(rs, mu.w, o[db][4 * g + 3]);
        }
    }

    // O^T += V_hat^T P^T
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int kc = 0; kc < 2; ++kc) {
        const int base = ((((kc * 4 + db) * 2 + kh) * 2) * 32 + col) * 16;
        const u4 lo = *reinterpret_cast<const u4*>(&sm.v[buf][base]);
        const u4 hi = *reinterpret_cast<const u4*>(&sm.v[buf][base + 512]);
        const v8i vop = {(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
        o[db] = mfma_f8(vop, pop[kc], o[db]);
      }

    l_run = alpha * l_run + rs;
    m_run = m_new;
    if (j + 1 < a.T) stash(buf ^ 1);
    __syncthreads();
  }

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
        uint32_t w0 = (uint32_t)f32_to_bf16(o[db][4 * g + 0] * sm.sv[c0 + 0] * inv_l) |
                      ((uint32_t)f32_to_bf16(o[db][4 * g + 1] * sm.sv[c0 + 1] * inv_l) << 16);
        uint32_t w1 = (uint32_t)f32_to_bf16(o[db][4 * g + 2] * sm.sv[c0 + 2] * inv_l) |
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
