// 8-bit VC-Attention forward on gfx950 matrix cores (Sec. 3.1 eq. tiled-low-bit-attention,
// Sec. 3.2 eq. vc-online-update, Sec. 3.3 eq. direct-fp8).
//
// One workgroup = 256 queries (two 128-row query blocks) of one (batch, head): eight waves of 32
// queries, two per SIMD. Both products are computed transposed so that a lane owns one query:
//   S^T = K_hat Q_hat^T   INT8 MFMA 32x32x32 (A = key rows from LDS, B = the wave's queries held
//                         in registers for the whole kernel);
//   O^T += V_hat^T P^T    FP8 MFMA 32x32x64 (A = residual codes from LDS, B = P codes).
// A lane's 16 results of a 32-key block are 16 keys of its own query, so the running row maximum
// is an in-register max plus one exchange with lane l^32, alpha and l are per-lane scalars, and the
// ExpCast-FP8 codes are already in the B-operand order of the FP8 product: byte s of lane half kh
// in key chunk kc is key 32(2kc + s/16) + 8((s%16)/4) + 4kh + s%4, the order in which the
// preprocessing stores V_hat.
//
// Ping-pong schedule. Each wave alternates a matrix phase M_j (value product and row sum of tile j,
// scores of tile j+1) and a vector phase V_j (running maximum, rescale and ExpCast codes of tile j).
// Waves 4..7 run one phase behind waves 0..3 and every phase ends at a workgroup barrier; waves w
// and w+4 share a SIMD, so on every SIMD one wave feeds the matrix cores while the other runs the
// softmax on the vector ALU.
//
// Per score the vector ALU does one int-to-float conversion, one fp32 fma and one
// round-to-nearest-even saturating byte conversion (the code is the one-rounding
// fma(float(acc), 8a, fl(fl(120 + beta) - 8m')) of the method's fp32 formula), plus half a max3.
// The probability row sum r_j is an all-ones E4M3 A operand times the P codes. Block means are
// restored in batches of 8 tiles: (r_j, m_j) is kept in LDS, and every 8 tiles
// O^T += M^T R with R_t = r_t 2^(m_t - m) is one bf16 matrix product pair (mu_t / s_V and R split
// into hi + lo bf16 parts, relative error ~2^-16). The rescale by alpha is skipped when no row
// maximum of the wave moved.
//
// Tiles go straight from memory into LDS (16 KB of K_hat, 16 KB of V_hat per tile, four buffers),
// issued as asm so that the compiler adds no waits of its own: each wave waits (vmcnt) for its own
// share of a tile pair before the barrier that precedes the pair's first use, and the copies of
// the next two pairs stay in flight. Half of V_j's operands are read into registers at the end of
// V_j, when the LDS port of that wave is otherwise idle. The steady-state loop is unrolled by four
// tiles so that every LDS access names its buffer statically. Tiles are visited in ascending order
// with the running maximum updated once per 128-key tile, the schedule on which the codes are
// defined.
#include <type_traits>

#include "vc_common.hpp"
#include "vc_internal.hpp"

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

namespace vc {

constexpr int FWD_WAVES = 8;
constexpr int FWD_THREADS = 64 * FWD_WAVES;
constexpr int FWD_QUERIES = 32 * FWD_WAVES;  // 256: two query blocks
constexpr int TILE_BYTES = BLK * D;          // 16384
constexpr int VBUF_BYTES = TILE_BYTES + 2 * D;  // V tile, then its 128 bf16 means
// s_waitcnt immediates (vmcnt in bits 3:0 and 15:14, the other counters left at their maxima)
constexpr int WAIT_VM0 = 0x3f70;
constexpr int WAIT_VM_PAIR = 0x3f75;    // vmcnt(5): the five copies of one pair may remain
constexpr int WAIT_VM_2PAIRS = 0x3f7a;  // vmcnt(10): the copies of two pairs may remain

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ v16i mfma_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mfma_f8(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// Copies from global memory straight into LDS: lane l moves `bytes` bytes from base + voff to
// LDS address lds + l * bytes. Issued as asm so that the compiler inserts no waits of its own for
// them: the schedule waits for its copies explicitly (vmcnt) before the barrier that precedes
// their first use.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(LDS_PTR(p)));
}
__device__ __forceinline__ void copy16_to_lds(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void copy4_to_lds(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1" ::"v"(voff), "s"(base), "s"(lds)
               : "memory", "m0");
}

// Workgroup barrier for the phase schedule. The wave's own LDS stores are complete before it
// (lgkmcnt(0)); the tile copies into LDS are waited for explicitly (vmcnt) by the caller, so the
// copies issued for later tiles stay in flight across it. The empty asm statements keep the
// compiler from moving memory accesses across, the scheduling barriers keep it from moving
// anything across.
__device__ __forceinline__ void wg_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
}

// Empty asm that reads and rewrites x: values computed in a phase stay in that phase (the compiler
// may not sink their computation past the barrier that ends it).
template <typename V>
__device__ __forceinline__ void pin(V& x) {
  asm volatile("" : "+v"(x));
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

// wait until at most n pairs' copies (5 each) of this wave are in flight
__device__ __forceinline__ void wait_pairs(int n) {
  if (n >= 2) __builtin_amdgcn_s_waitcnt(WAIT_VM_2PAIRS);
  else if (n == 1) __builtin_amdgcn_s_waitcnt(WAIT_VM_PAIR);
  else __builtin_amdgcn_s_waitcnt(WAIT_VM0);
}

template <int PMODE>
__global__ __launch_bounds__(FWD_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_fwd(FwdArgs a) {
  // four tile buffers: K_0 in buffer 0, pair p = (K_{p+1}, V_p with its block means) in buffer (p+1) mod 4
  __shared__ __attribute__((aligned(16))) uint8_t kb0[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb1[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb2[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb3[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb0[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb1[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb2[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb3[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint16_t ub[2][2][D][8];        // [chunk parity][hi, lo][channel][slot]
  __shared__ __attribute__((aligned(16))) float2 rm[FWD_WAVES][32][8];   // (r_t, m_t) per query, slot t % 8
  __shared__ float svs[D], inv_svs[D];

  const int qt = blockIdx.x, bh = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kh = lane >> 5, col = lane & 31;
  const bool lead = wave < FWD_WAVES / 2;  // waves 0..3 lead, 4..7 (same SIMDs) follow one phase behind
  const int T = a.T;
  const size_t tile0 = (size_t)bh * T;

  // the wave's 32 queries (query block 2 qt + wave / 4, rows 32 (wave % 4) ..) as the B operand
  const int qblock = min(2 * qt + (wave >> 2), T - 1);
  const int8_t* qblk = a.q + (tile0 + qblock) * TILE_BYTES;
  v4i qop[4];
#pragma unroll
  for (int dc = 0; dc < 4; ++dc)
    qop[dc] = *reinterpret_cast<const v4i*>(qblk + (((wave & 3) * 4 + dc) * 2 + kh) * 512 + col * 16);
  const float sq = a.q_scale[tile0 + qblock];

  const int mc = tid & (D - 1);
  if (tid < D) {
    const float sv = a.v_scale[(size_t)bh * D + tid];
    svs[tid] = sv;
    inv_svs[tid] = 1.f / sv;
  }
  reinterpret_cast<u4*>(&ub[0][0][0][0])[tid] = u4{0, 0, 0, 0};  // 512 x 16 B: the whole array

  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + tile0 * TILE_BYTES;
  const uint8_t* vbase = a.v + tile0 * TILE_BYTES;
  const uint8_t* mbase = reinterpret_cast<const uint8_t*>(a.v_mean + tile0 * D) + 32 * wave;
  // K_0: two 1 KB copies per wave
  auto load_k0 = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int off = (u * FWD_WAVES + wave) * 1024;
      copy16_to_lds(kbase + off, lane * 16, lds_addr(kb0 + off));
    }
  };
  // copy k (0..4) of pair p: two 1 KB pieces of K_{p+1} (clamped to the last tile), two of V_p,
  // 32 bytes of V_p's means. Every wave issues exactly five copies per pair, the number the
  // waits count.
  auto load_part = [&](int k, int p, uint8_t* kd, uint8_t* vd) __attribute__((always_inline)) {
    if (k < 4) {
      const uint8_t* src = k < 2 ? kbase + (size_t)min(p + 1, T - 1) * TILE_BYTES : vbase + (size_t)p * TILE_BYTES;
      uint8_t* dst = k < 2 ? kd : vd;
      const int off = ((k & 1) * FWD_WAVES + wave) * 1024;
      copy16_to_lds(src + off, lane * 16, lds_addr(dst + off));
    } else if (lane < 8) {
      copy4_to_lds(mbase + (size_t)p * 2 * D, 4 * lane, lds_addr(vd + TILE_BYTES + 32 * wave));
    }
  };
  auto load_pair = [&](int p, uint8_t* kd, uint8_t* vd) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < 5; ++k) load_part(k, p, kd, vd);
  };
  // K scales through the scalar cache
  const __attribute__((address_space(4))) float* kscale =
      (const __attribute__((address_space(4))) float*)(a.k_scale + tile0);
  // mu_j / s_V as bf16 hi + lo into slot j % 8 of chunk parity (j / 8) % 2, from the means behind
  // V_j in vt (leaders only: threads 128..255 store the same values as threads 0..127)
  auto stash_mean = [&](int j, const uint8_t* vt) __attribute__((always_inline)) {
    if (a.smooth_v) {
      const float u = bf16_to_f32(reinterpret_cast<const uint16_t*>(vt + TILE_BYTES)[mc]) * inv_svs[mc];
      const uint16_t hi = f32_to_bf16(u);
      ub[(j >> 3) & 1][0][mc][j & 7] = hi;
      ub[(j >> 3) & 1][1][mc][j & 7] = f32_to_bf16(u - bf16_to_f32(hi));
    }
  };

  v16f o[4];
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;
  const v8i ones = {0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838, 0x38383838};
  // s: scores of the tile whose codes are computed next; after the vector phase s[0] holds that
  // tile's ExpCast codes (the two v8i B operands of the value product)
  v16i s[4];
  v8i vops[4];              // first half of the V_j operands, read at the end of V_j for M_j
  float rsum = 0.f;         // row sum of the tile whose value product was issued last
  float ksc = 0.f;          // scale of the K tile whose scores are in s
  float2* rm_q = &rm[wave][col][0];

  // O^T += M^T R for the tiles of chunk parity `par` whose slot is <= last_slot, R_t = r_t 2^(m_t - m)
  auto flush_means = [&](int par, int last_slot) __attribute__((always_inline)) {
    bf16x8 b;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float2 e = rm_q[t];
      const float R = t <= last_slot ? e.x * __builtin_amdgcn_exp2f(e.y - m_run) : 0.f;
      const uint16_t hi = f32_to_bf16(R);
      const uint16_t v = kh == 0 ? hi : f32_to_bf16(R - bf16_to_f32(hi));
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
  };

  // r of tile jp (computed by the matrix phase before, at the running maximum m_run) into l and
  // slot jp % 8 of (r, m)
  auto fold_rowsum = [&](int jp) __attribute__((always_inline)) {
    l_run += rsum;
    rm_q[jp & 7] = make_float2(rsum, m_run);
  };

  // V_j operand n of the value product (A operand: residual codes, 32 channels x 64 keys)
  auto load_vop = [&](const uint8_t* vt, int n) __attribute__((always_inline)) -> v8i {
    const int kc = n >> 2, db = n & 3;
    const int base = ((((kc * 4 + db) * 2 + kh) * 2) * 32 + col) * 16;
    const u4 lo = *reinterpret_cast<const u4*>(vt + base);
    const u4 hi = *reinterpret_cast<const u4*>(vt + base + 512);
    return v8i{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };
  auto prefetch_v = [&](const uint8_t* vt) __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);  // after the codes: the scores' registers are free by then
#pragma unroll
    for (int n = 0; n < 4; ++n) vops[n] = load_vop(vt, n);
  };

  // matrix phase M_j: value product and row sum of tile j (codes in s[0], operands in vops), scores
  // of tile j+1 (K_{j+1} in kt, read two pieces behind each value product), then the means of chunk
  // j/8 - 1 once j is a multiple of 8. hook(n), n = 0..4, issues copy n of a later pair between the
  // products. PVC / QKC / MASKC (std::integral_constant): value product, scores, ragged tile j+1.
  auto mphase_m = [&](auto PVC, auto QKC, auto MASKC, int j, const uint8_t* kt, const uint8_t* vt, auto hook) __attribute__((always_inline)) {
    constexpr bool pv = decltype(PVC)::value, qk = decltype(QKC)::value;
    v4i kops[16];
    auto load_k = [&](int n) __attribute__((always_inline)) {
      const int dc = n >> 2, kb = n & 3;
      kops[n] = *reinterpret_cast<const v4i*>(kt + ((kb * 4 + dc) * 2 + kh) * 512 + col * 16);
    };
    if (pv) {
      const v8i p0 = __builtin_shufflevector(s[0], s[0], 0, 1, 2, 3, 4, 5, 6, 7);
      const v8i p1 = __builtin_shufflevector(s[0], s[0], 8, 9, 10, 11, 12, 13, 14, 15);
      v8i vops2[4];
#pragma unroll
      for (int n = 0; n < 4; ++n) vops2[n] = load_vop(vt, 4 + n);
      v16f rs = {};
      rs = mfma_f8(ones, p0, rs);
      rs = mfma_f8(ones, p1, rs);
#pragma unroll
      for (int n = 0; n < 8; ++n) {
        const int kc = n >> 2, db = n & 3;
        o[db] = mfma_f8(n < 4 ? vops[n] : vops2[n - 4], kc == 0 ? p0 : p1, o[db]);
        if (qk) {
          load_k(2 * n);
          load_k(2 * n + 1);
        }
        if (n < 5) hook(n);
      }
      rsum = rs[0];
    } else {
#pragma unroll
      for (int n = 0; n < 16; ++n) {
        if (qk) load_k(n);
        if (n < 5) hook(n);
      }
    }
    if (qk) {
      ksc = kscale[j + 1];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = 0;
#pragma unroll
      for (int n = 0; n < 16; ++n) {
        const int dc = n >> 2, kb = n & 3;
        s[kb] = mfma_i8(kops[n], qop[dc], s[kb]);
      }
      if (decltype(MASKC)::value) mask_tile(s, kh, a.N - (T - 1) * BLK);
    }
    if (pv && qk) {
      __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
#pragma unroll
      for (int n = 0; n < 8; ++n) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);
    }
    if (pv && a.smooth_v && j >= 8 && (j & 7) == 0) flush_means(((j >> 3) - 1) & 1, 7);
  };

  // vector phase V_j: fold r_{j-1}; running maximum and alpha of tile j; rescale; codes of tile j
  // into s[0]. LASTC (std::integral_constant): tile j is the ragged last tile.
  auto vphase = [&](auto LASTC, int j) __attribute__((always_inline)) {
    constexpr bool last = decltype(LASTC)::value;
    if (j >= 1) fold_rowsum(j - 1);
    const float a_s = (sq * ksc) * a.kappa;  // the oracle's order: fl(fl(s_q s_k) kappa)
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
    if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      l_run *= alpha;
    }
    const float a8 = 8.f * a_s;
    const float bias = a.cbias - 8.f * m_new;
    v8i p[2];
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
    s[0] = __builtin_shufflevector(p[0], p[1], 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15);
  };

  const std::integral_constant<bool, false> NO;
  const std::integral_constant<bool, true> YES;
  auto nohook = [](int) {};

  // end of a phase: the phase's results are final before the workgroup barrier, and the next
  // phase's work starts after it
  auto pin_state = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < 4; ++db) pin(o[db]);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) pin(s[kb]);
    pin(l_run);
    pin(m_run);
    pin(rsum);
    pin(ksc);
  };
  // wait: -1 none, else the number of this wave's pairs that may stay in flight
  auto end_phase = [&](int wait) __attribute__((always_inline)) {
    pin_state();
    if (wait >= 0) wait_pairs(wait);
    wg_barrier();
    pin_state();
  };

  // Every wave runs the phase sequence M_{-1}, V_0, M_0, V_1, ..., V_{T-1}, M_{T-1}, F with a
  // barrier after each phase; the followers pass one extra barrier before their first phase and
  // the leaders one after their last, so a follower's phase k meets a leader's phase k+1 (global
  // phase 2j+1 holds the leaders' V_j and the followers' M_{j-1}). Pair p is read from global
  // phase 2p+1 on (the leaders' V_p reads V_p's operands and means, M_p reads K_{p+1}) until 2p+3,
  // so it must have landed in every wave's share by the barrier ending global phase 2p: the leaders
  // wait after M_{p-1}, the followers after V_{p-1}. A wave issues its share of pair p during its
  // M_{p-3}, between the value products; the pair's buffer was last read by pair p-4 in global
  // phase 2p-5.
  const bool t2 = T > 1, t3 = T > 2;
  __builtin_amdgcn_s_waitcnt(WAIT_VM0);  // the compiler's own loads have landed before any copy
  load_k0();
  load_pair(0, kb1, vb1);
  if (t2) load_pair(1, kb2, vb2);
  wait_pairs(t2 ? 2 : 1);  // K_0
  wg_barrier();
  if (!lead) {
    wait_pairs(t2 ? 1 : 0);  // pair 0
    wg_barrier();
  }
  // M_{-1}: scores of tile 0; pair 2 copied
  auto hook_m1 = [&](int k) __attribute__((always_inline)) {
    if (t3) load_part(k, 2, kb3, vb3);
  };
  if (T == 1) mphase_m(NO, YES, YES, -1, kb0, vb0, hook_m1);
  else mphase_m(NO, YES, NO, -1, kb0, vb0, hook_m1);
  end_phase(lead ? (int)t2 + (int)t3 : -1);  // leaders: pair 0
  // V_0
  if (T == 1) vphase(YES, 0);
  else vphase(NO, 0);
  prefetch_v(vb1);
  end_phase(lead ? -1 : (int)t3);  // followers: pair 1

  // steady-state tile step i (pair i+3 exists, i + 3 <= T - 1): M_i on the operands of V_i and
  // K_{i+1} in buffer (ks) = (i+1) mod 4, copying pair i+3 into (kd, vd) = i mod 4; V_{i+1} (leaders
  // stash mean i from vs) and the operands of V_{i+1} from vn = (i+2) mod 4
  auto steady = [&](int i, uint8_t* kd, uint8_t* vd, const uint8_t* ks, const uint8_t* vs, const uint8_t* vn) __attribute__((always_inline)) {
    auto hook = [&](int k) __attribute__((always_inline)) { load_part(k, i + 3, kd, vd); };
    mphase_m(YES, YES, NO, i, ks, vs, hook);
    end_phase(lead ? 2 : -1);  // leaders: pair i+1
    if (lead) stash_mean(i, vs);
    vphase(NO, i + 1);
    prefetch_v(vn);
    end_phase(lead ? -1 : 1);  // followers: pair i+2
  };
  int i = 0;
  for (; i + 7 <= T; i += 4) {
    steady(i, kb0, vb0, kb1, vb1, vb2);
    steady(i + 1, kb1, vb1, kb2, vb2, vb3);
    steady(i + 2, kb2, vb2, kb3, vb3, vb0);
    steady(i + 3, kb3, vb3, kb0, vb0, vb1);
  }
  if (i + 4 <= T) {
    steady(i, kb0, vb0, kb1, vb1, vb2);
    ++i;
    if (i + 4 <= T) {
      steady(i, kb1, vb1, kb2, vb2, vb3);
      ++i;
      if (i + 4 <= T) {
        steady(i, kb2, vb2, kb3, vb3, vb0);
        ++i;
      }
    }
  }
  // tail: no copies issued any more, every copy waited for
  auto kbuf = [&](int b) __attribute__((always_inline)) -> const uint8_t* {
    return b == 0 ? kb0 : (b == 1 ? kb1 : (b == 2 ? kb2 : kb3));
  };
  auto vbuf = [&](int b) __attribute__((always_inline)) -> const uint8_t* {
    return b == 0 ? vb0 : (b == 1 ? vb1 : (b == 2 ? vb2 : vb3));
  };
  // tile steps T-3 (if it had no copy to issue), T-2 (scores and codes of the ragged last tile)
  // and T-1 (its value product and the final means)
  if (i == T - 3) {
    const int b = (i + 1) & 3;
    mphase_m(YES, YES, NO, i, kbuf(b), vbuf(b), nohook);
    end_phase(0);
    if (lead) stash_mean(i, vbuf(b));
    vphase(NO, i + 1);
    prefetch_v(vbuf((i + 2) & 3));
    end_phase(0);
    ++i;
  }
  if (i == T - 2) {
    const int b = (i + 1) & 3;
    mphase_m(YES, YES, YES, i, kbuf(b), vbuf(b), nohook);
    end_phase(0);
    if (lead) stash_mean(i, vbuf(b));
    vphase(YES, i + 1);
    prefetch_v(vbuf((i + 2) & 3));
    end_phase(0);
    ++i;
  }
  {
    const int b = T & 3;
    mphase_m(YES, NO, NO, T - 1, kbuf(b), vbuf(b), nohook);
    end_phase(0);
    if (lead) stash_mean(T - 1, vbuf(b));
    fold_rowsum(T - 1);
    if (a.smooth_v) flush_means(((T - 1) >> 3) & 1, (T - 1) & 7);
    end_phase(0);
  }
  if (lead) wg_barrier();

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
