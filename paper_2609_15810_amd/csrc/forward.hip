// 8-bit VC-Attention forward on gfx950 matrix cores (Sec. 3.1 eq. tiled-low-bit-attention,
// Sec. 3.2 eq. vc-online-update, Sec. 3.3 eq. direct-fp8).
//
// One workgroup = 256 queries (two 128-row query blocks) of one (batch, head): eight waves of 32
// queries, two waves per SIMD, so that one wave's matrix-core work can overlap the other wave's
// softmax on the vector ALU. Both products are computed transposed so that a lane owns one query:
//   S^T = K_hat Q_hat^T   INT8 MFMA 32x32x32 (A = key rows from LDS, B = the wave's queries held
//                         in registers for the whole kernel);
//   O^T += V_hat^T P^T    FP8 MFMA 32x32x64 (A = residual codes from LDS, B = P codes).
// A lane's 16 results of a 32-key block are 16 keys of its own query, so the running row maximum
// is an in-register max plus one exchange with lane l^32, alpha and l are per-lane scalars, and the
// ExpCast-FP8 codes are already in the B-operand order of the FP8 product: byte s of lane half kh
// in key chunk kc is key 32(2kc + s/16) + 8((s%16)/4) + 4kh + s%4, the order in which the
// preprocessing stores V_hat.
//
// Per score the vector ALU does one int-to-float conversion, one fp32 fma and one
// round-to-nearest-even saturating byte conversion (the code is the one-rounding
// fma(float(acc), 8a, fl(fl(120 + beta) - 8m')) of the method's fp32 formula), plus half a max3.
// Everything else is moved off the vector ALU or amortised:
//   - the probability row sum r is an all-ones E4M3 A operand times the P codes;
//   - block means are restored in batches of 8 tiles: r_j (rescaled with A) is kept per lane and
//     every 8 tiles O^T += M^T R is one bf16 matrix product with mu_j / s_V and r split into
//     hi + lo bf16 parts (hi*hi + hi*lo + lo*hi, relative error ~2^-16);
//   - the rescale of A by alpha is skipped when no row maximum of the wave moved.
// K_hat and V_hat tiles (16 KB each) go straight from memory into a double-buffered LDS region (no
// staging registers); the next tile is in flight while the current one is consumed. Tiles are
// visited in ascending order with the running maximum updated once per 128-key tile, the schedule
// on which the codes are defined.
#include <type_traits>

#include "vc_common.hpp"
#include "vc_internal.hpp"

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

namespace vc {

constexpr int FWD_WAVES = 8;
constexpr int FWD_THREADS = 64 * FWD_WAVES;
constexpr int FWD_QUERIES = 32 * FWD_WAVES;  // 256: two query blocks
constexpr int TILE_BYTES = BLK * D;          // 16384

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

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

template <int PMODE>
__global__ __launch_bounds__(FWD_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd(FwdArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t kb0[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb1[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb0[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb1[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint16_t ub[2][2][D][8];  // [chunk parity][hi, lo][channel][slot]
  __shared__ float svs[D];

  const int qt = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kh = lane >> 5, col = lane & 31;
  const int T = a.T;
  const size_t tile0 = (size_t)bh * T;

  // the wave's 32 queries (query block qt*WAVES/4 + wave/4, rows 32*(wave%4) ..) as the B operand
  const int qblock = min(qt * (FWD_WAVES / 4) + (wave >> 2), T - 1);
  const int8_t* qblk = a.q + (tile0 + qblock) * TILE_BYTES;
  v4i qop[4];
#pragma unroll
  for (int dc = 0; dc < 4; ++dc)
    qop[dc] = *reinterpret_cast<const v4i*>(qblk + (((wave & 3) * 4 + dc) * 2 + kh) * 512 + col * 16);
  const float sq = a.q_scale[tile0 + qblock];

  const float inv_sv = 1.f / a.v_scale[(size_t)bh * D + (tid & (D - 1))];
  if (tid < D) svs[tid] = a.v_scale[(size_t)bh * D + tid];

  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + tile0 * TILE_BYTES;
  const uint8_t* vbase = a.v + tile0 * TILE_BYTES;
  // one 16 KB tile straight into LDS: each wave moves TILE_BYTES / FWD_WAVES bytes
  auto load_tile = [&](const uint8_t* src, uint8_t* dst) {
#pragma unroll
    for (int u = 0; u < TILE_BYTES / (1024 * FWD_WAVES); ++u) {
      const int off = (u * FWD_WAVES + wave) * 1024;
      __builtin_amdgcn_global_load_lds(src + off + lane * 16, LDS_PTR(dst + off), 16, 0, 0);
    }
  };
  // block means: thread tid handles channel tid & 127; the threads 128.. compute and store the same
  // value as their partner (a duplicate store of equal data), so the tile loop has no divergent branch
  const int mc = tid & (D - 1);
  const float mean_gate = a.smooth_v ? 1.f : 0.f;
  float mu_reg = 0.f;
  auto load_mean = [&](int j) { mu_reg = bf16_to_f32(a.v_mean[(tile0 + j) * D + mc]); };
  auto stash_mean = [&](int j) {  // mu_j / s_V as bf16 hi + lo in slot j of its chunk
    const float u = mu_reg * inv_sv * mean_gate;
    const uint16_t hi = f32_to_bf16(u);
    ub[(j >> 3) & 1][0][mc][j & 7] = hi;
    ub[(j >> 3) & 1][1][mc][j & 7] = f32_to_bf16(u - bf16_to_f32(hi));
  };

  v16f o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float R[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) R[t] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const v8i ones = {0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838};

  // O^T += M^T R for the 8 tiles of chunk `par` (bf16 hi/lo products), then R = 0
  auto flush_means = [&](int par) {
    bf16x8 b;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const uint16_t hi = f32_to_bf16(R[t]);
      const uint16_t v = kh == 0 ? hi : f32_to_bf16(R[t] - bf16_to_f32(hi));
      b[t] = __builtin_bit_cast(__bf16, v);
    }
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      const int c = 32 * db + col;
      const bf16x8 a_hi = *reinterpret_cast<const bf16x8*>(&ub[par][0][c][0]);
      bf16x8 a_lo = *reinterpret_cast<const bf16x8*>(&ub[par][1][c][0]);
      if (kh) a_lo = bf16x8{};
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_hi, b, o[db], 0, 0, 0);
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_lo, b, o[db], 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) R[t] = 0.f;
  };

  v16i s[4];  // scores of the current tile
  v8i p[2];   // its probability codes (B operand of the FP8 value product)

  auto add_rowsum = [&](int jp, const v16f& rs) {
    const float r = rs[0];
    l_run += r;
    const int slot = jp & 7;
#pragma unroll
    for (int t = 0; t < 8; ++t) R[t] = t == slot ? r : R[t];
    if (a.smooth_v && slot == 7) flush_means((jp >> 3) & 1);
  };

  // tile j: scores, codes, row sum, rescale, value product. K_j / V_j are in buffer j&1, tile j+1
  // is in flight into the other buffer. LASTC: std::integral_constant, true for the (possibly
  // ragged) last tile only, so the steady-state loop carries no masking code.
  auto step = [&](auto LASTC, int j, const uint8_t* kt, const uint8_t* vt) {
    constexpr bool last = decltype(LASTC)::value;
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
    if (last) mask_tile(s, kh, a.N - j * BLK);
    const float a_s = (sq * a.k_scale[tile0 + j]) * a.kappa;
    int mk[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      int m = max(s[kb][0], s[kb][1]);
#pragma unroll
      for (int r = 2; r < 16; r += 2) m = max(max(m, s[kb][r]), s[kb][r + 1]);
      mk[kb] = m;
    }
    int mx = max(max(mk[0], mk[1]), max(mk[2], mk[3]));
    mx = max(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, (float)mx * a_s);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    const float a8 = 8.f * a_s;
    const float bias = a.cbias - 8.f * m_new;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int d4 = 0; d4 < 4; ++d4) {
        uint32_t w = 0;
        if (PMODE == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            w = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_fmaf((float)s[kb][4 * d4 + q], a8, bias), q, w);
        } else {
          float pe[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) pe[q] = __builtin_amdgcn_exp2f((float)s[kb][4 * d4 + q] * a_s - m_new) * 256.f;
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(pe[0], pe[1], 0, false);
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(pe[2], pe[3], (int)w, true);
        }
        p[kb >> 1][4 * (kb & 1) + d4] = (int)w;
      }
    if (last) clear_padded(p, kh, a.N - j * BLK);
    v16f rs = {};
    rs = mfma_f8(ones, p[0], rs);
    rs = mfma_f8(ones, p[1], rs);
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
#pragma unroll
      for (int t = 0; t < 8; ++t) R[t] *= alpha;
      l_run *= alpha;
    }
    pv_tile(vt, p, kh, col, o);
    add_rowsum(j, rs);
    __builtin_amdgcn_s_waitcnt(0x3f70);  // vmcnt(0): tile j+1 and mean j+1 have landed
    stash_mean(j + 1);
    __syncthreads();
    if (j + 2 < T) {
      load_tile(kbase + (size_t)(j + 2) * TILE_BYTES, const_cast<uint8_t*>(kt));
      load_tile(vbase + (size_t)(j + 2) * TILE_BYTES, const_cast<uint8_t*>(vt));
      load_mean(j + 2);
    }
  };

  load_tile(kbase, kb0);
  load_tile(vbase, vb0);
  load_mean(0);
  __builtin_amdgcn_s_waitcnt(0x3f70);
  stash_mean(0);
  __syncthreads();
  if (T > 1) {
    load_tile(kbase + TILE_BYTES, kb1);
    load_tile(vbase + TILE_BYTES, vb1);
    load_mean(1);
  }
  const std::integral_constant<bool, false> F;
  const std::integral_constant<bool, true> Tr;
  int j = 0;
  for (; j + 2 < T; j += 2) {
    step(F, j, kb0, vb0);
    step(F, j + 1, kb1, vb1);
  }
  if (T - j == 2) {
    step(F, j, kb0, vb0);
    step(Tr, j + 1, kb1, vb1);
  } else {
    step(Tr, j, kb0, vb0);
  }
  if (a.smooth_v && ((T - 1) & 7) != 7) flush_means(((T - 1) >> 3) & 1);

  // epilogue: O = A s_V / l, bf16, row q written to token q_perm[q] (or q)
  const int q = qt * FWD_QUERIES + wave * 32 + col;
  if (q < a.N) {
    const float inv_l = 1.f / l_run;
    const int qo = a.q_perm ? clamp_index(a.q_perm[(size_t)bh * a.N + q], a.N) : q;
    uint16_t* orow = a.O + ((size_t)bh * a.N + qo) * D;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int c0 = 32 * db + 8 * g + 4 * kh;
        const uint32_t w0 = (uint32_t)f32_to_bf16(o[db][4 * g + 0] * svs[c0 + 0] * inv_l) |
                            ((uint32_t)f32_to_bf16(o[db][4 * g + 1] * svs[c0 + 1] * inv_l) << 16);
        const uint32_t w1 = (uint32_t)f32_to_bf16(o[db][4 * g + 2] * svs[c0 + 2] * inv_l) |
                            ((uint32_t)f32_to_bf16(o[db][4 * g + 3] * svs[c0 + 3] * inv_l) << 16);
        *reinterpret_cast<uint2*>(orow + c0) = make_uint2(w0, w1);
      }
  }
}

hipError_t launch_forward(const FwdArgs& a, int BH, hipStream_t s) {
  const dim3 grid((a.N + FWD_QUERIES - 1) / FWD_QUERIES, BH);
  if (a.p_mode == 0) attn_fwd<0><<<grid, FWD_THREADS, 0, s>>>(a);
  else attn_fwd<1><<<grid, FWD_THREADS, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace vc
