// 8-bit VC-Attention forward on gfx950 matrix cores (Sec. 3.1 eq. tiled-low-bit-attention,
// Sec. 3.2 eq. vc-online-update, Sec. 3.3 eq. direct-fp8).
//
// One workgroup = 256 queries (two 128-row query blocks) of one (batch, head): eight waves of 32
// queries, two per SIMD. Both products are computed transposed so that a lane owns one query:
//   S^T = K_hat Q_hat^T   INT8 MFMA 32x32x32 (A = key rows from LDS, B = the wave's queries held
//                         in registers for the whole kernel);
//   O^T += V_hat^T P^T    FP8 MFMA 32x32x64 (A = residual codes from LDS, B = P codes).
// A lane's 16 results of a 32-key block are 16 keys of its own query, so the running row maximum
// is an in-register max plus one exchange with lane l^32 (v_permlane32_swap), alpha and l are
// per-lane scalars, and the ExpCast-FP8 codes are already in the B-operand order of the FP8
// product: byte s of lane half kh in key chunk kc is key 32(2kc + s/16) + 8((s%16)/4) + 4kh + s%4,
// the order in which the preprocessing stores V_hat.
//
// Software pipeline inside each wave. Iteration j issues the value product of tile j (its codes
// were formed in iteration j-1), forms the running maximum and the codes of tile j+1, and issues
// the scores of tile j+2, in regions that each pair matrix work with vector work of about the same
// length (scheduling barriers keep the regions in order; the codes of key block kb of tile j+1
// are formed before the scores of block kb of tile j+2 overwrite its registers). The matrix cores
// thus run the value and score products of one wave while its vector ALU forms codes; the two
// waves of a SIMD share both.
//
// Per score the vector ALU does one int-to-float conversion, one fp32 fma (the code is the
// one-rounding fma(float(acc), 8a, fl(fl(120 + beta) - 8m')) of the method's fp32 formula, evaluated
// scaled by 2^-24 with the clamp at 0 folded in), half an fp16 pair conversion (which rounds to the
// nearest-even integer code and leaves it in the low bits) and a quarter of a byte permute, plus
// half a max3.
// The probability row sum r_j is one FP8 16x16x128 product per 64 keys whose A operand holds ones
// only in rows 0, 4, 8 and 12 (so that lane l receives r of its own query). Block means are
// restored in batches of 8 tiles: (r_j, m_j) is kept in LDS, and every 8 tiles O^T += M^T R with
// R_t = r_t 2^(m_t - m) is one bf16 matrix product pair (mu_t / s_V and R split into hi + lo bf16
// parts, all four cross terms, relative error ~2^-16). The rescale by alpha is skipped when no row
// maximum of the wave moved.
//
// Tiles go straight from memory into LDS (16 KB of K_hat, 16 KB of V_hat per tile, four buffers
// each), issued as asm so that the compiler adds no waits of its own: pair p = (K_{p+2}, V_p with
// its block means) is copied during iteration p-3, each wave waits (vmcnt) for its own share of
// pair p+1 before the barrier that ends iteration p, and the next two pairs stay in flight. The
// steady-state loop is unrolled by four iterations so that every LDS access names its buffer
// statically. Tiles are visited in ascending order with the running maximum updated once per
// 128-key tile, the schedule on which the codes are defined.
//
// FP8 Q/K variant (E4M3 per 128-row block, for matrix units without INT8): the scores come from
// two FP8 32x32x64 products per 32-key block (each lane 32 channels of its row), already fp32.
//
// 4-bit variant (OCP MXFP4 Q and K): the scores come from the scaled FP4 product
// v_mfma_scale_f32_32x32x64_f8f6f4 (two per 32-key block), each lane's E8M0 byte scaling its
// 32-channel block, so S^T arrives in fp32 with the block scales applied and the score scale of
// the codes is kappa alone. A K tile is 8 KB of packed codes followed by its 512 scale bytes;
// everything after the scores is shared with the 8-bit path.
#include <type_traits>

#include "vc_common.hpp"
#include "vc_internal.hpp"

#define LDS_PTR(p) ((__attribute__((address_space(3))) void*)(p))

namespace vc {

constexpr int NW = 8;             // waves per workgroup, 32 queries each (two per SIMD)
constexpr int NXCD = 8;           // accelerator complex dies (each with its own L2)
constexpr int NTH = 64 * NW;
constexpr int NQ = 32 * NW;
constexpr int TILE_BYTES = BLK * D;
constexpr int VBUF_BYTES = TILE_BYTES + 2 * D;
constexpr int KCOPIES = TILE_BYTES / 1024 / NW;  // 1 KB copies per wave per tile (V; INT8 K)
constexpr int PAIR_COPIES = 2 * KCOPIES + 1;     // K and V pieces + the means
constexpr int MX_CODE_BYTES = TILE_BYTES / 2;    // packed E2M1 codes of a 128-key tile
constexpr int MX_SCALE_BYTES = BLK * D / 32;     // its E8M0 scale bytes, one per 32 channels
static_assert(MX_CODE_BYTES / 1024 / NW == 1 && MX_SCALE_BYTES / NW <= 4 * 64,
              "MXFP4 K tiles move as one 1 KB copy of codes and one 4-byte-per-lane copy of scales per wave");
static_assert(MX_CODE_BYTES + MX_SCALE_BYTES <= TILE_BYTES, "an MXFP4 K tile fits a K buffer");
constexpr int MEAN_LANES = 64 / NW;              // lanes copying 4 bytes of means each

// s_waitcnt immediate for vmcnt(n) (bits 3:0 and 15:14), the other counters left at their maxima
constexpr int vm_wait(int n) { return 0x3f70 | (n & 0xf) | ((n >> 4) << 14); }
// wait until at most n pairs' copies of this wave are in flight
__device__ __forceinline__ void wait_pairs(int n) {
  if (n >= 2) __builtin_amdgcn_s_waitcnt(vm_wait(2 * PAIR_COPIES));
  else if (n == 1) __builtin_amdgcn_s_waitcnt(vm_wait(PAIR_COPIES));
  else __builtin_amdgcn_s_waitcnt(vm_wait(0));
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float v4f __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v16i mfma_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mfma_f8(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}
__device__ __forceinline__ v4f mfma_f8_16(v8i a, v8i b, v4f c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// max of v over lanes l and l^32 (the two key halves of a query)
__device__ __forceinline__ int half_max(int v) {
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return max(max(v, (int)r[0]), (int)r[1]);
}
// fp32 version through the order-preserving map of fp32 bit patterns onto int32 (negative values
// get their magnitude bits flipped; the map is its own inverse). Written this way because
// fmaxf over the two outputs of the swap has been compiled into a max over one of them only.
__device__ __forceinline__ float half_max(float v) {
  const int b = __builtin_bit_cast(int, v);
  const int m = half_max(b ^ ((b >> 31) & 0x7fffffff));
  return __builtin_bit_cast(float, m ^ ((m >> 31) & 0x7fffffff));
}
__device__ __forceinline__ int smax(int a, int b) { return max(a, b); }
__device__ __forceinline__ float smax(float a, float b) { return fmaxf(a, b); }
__device__ __forceinline__ int smax3(int a, int b, int c) { return max(max(a, b), c); }
__device__ __forceinline__ float smax3(float a, float b, float c) { return fmaxf(fmaxf(a, b), c); }

// Scaled FP4 x FP4 product (cbsz = blgp = 4): a, b hold 32 E2M1 codes per lane (one 32-channel
// block of row / column l%32, channel block l/32 of the 64), scaled by byte OA of sa and byte OB
// of sb (E8M0)
template <int OA, int OB>
__device__ __forceinline__ v16f mfma_f4(v4i a, v4i b, v16f c, int sa, int sb) {
  const v8i a8 = __builtin_shufflevector(a, a, 0, 1, 2, 3, -1, -1, -1, -1);
  const v8i b8 = __builtin_shufflevector(b, b, 0, 1, 2, 3, -1, -1, -1, -1);
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, OA, sa, OB, sb);
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

// Workgroup barrier. The wave's own LDS stores are complete before it (lgkmcnt(0)); the tile
// copies into LDS are waited for explicitly (vmcnt) by the caller, so the copies issued for later
// tiles stay in flight across it. The empty asm statements keep the compiler from moving memory
// accesses across, the scheduling barriers keep it from moving anything across.
__device__ __forceinline__ void wg_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::: "memory");
}

// Empty asm that reads and rewrites x: x is formed before this point (a pure value would
// otherwise be computed next to its first use).
template <typename V>
__device__ __forceinline__ void pin(V& x) {
  asm volatile("" : "+v"(x));
}

// Padded keys of the last tile (key >= kvalid): the lowest score before the softmax ...
template <typename SV>
__device__ __forceinline__ void mask_tile(SV (&s)[4], int kh, int kvalid) {
  using E = std::remove_reference_t<decltype(s[0][0])>;
  constexpr E lowest = std::is_same_v<E, float> ? (E)-INFINITY : (E)INT_MIN;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (32 * kb + 8 * (r >> 2) + 4 * kh + (r & 3) >= kvalid) s[kb][r] = lowest;
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

// The clip of eq. direct-fp8 at code 120. The fma that forms the code of a score s <= M (the
// tile's largest) is at most cbias + 8(M a - fl(M a)) + |fl(cbias - 8m') - (cbias - 8m')|
// <= cbias + 4 ulp(m') + ulp(fl(cbias - 8m')) / 2 with cbias = fl(120 + beta) <= 120
// (-1 <= beta <= 0). For |m'| < 2^16 (log2 units) that is below 120 + 2^-4, so no code exceeds
// 120; a wave whose row maxima reach 2^16 clips its codes bytewise (a branch that scores of such
// size take). For |m'| < 2^27 it is below 217, so the codes still fit the byte the fp16
// conversion leaves (below 256) and the clip restores eq. direct-fp8. A row whose running
// maximum reaches 2^27 (the first or the last tile's: the running maximum is monotone) is
// outside that domain and its output is written as NaN.
constexpr float WIDE_MAX = 65536.f;
constexpr float DOMAIN_MAX = 134217728.f;
__device__ __forceinline__ void clip_codes(v8i (&pn)[2]) {
#pragma unroll
  for (int kc = 0; kc < 2; ++kc)
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const uint32_t u = (uint32_t)pn[kc][w];
      uint32_t r = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) r |= min((u >> (8 * b)) & 0xffu, 120u) << (8 * b);
      pn[kc][w] = (int)r;
    }
}

// DUMP: also write the probability codes of every tile to a.p_codes (a debugging variant; the
// stores wait for all copies in flight, so it runs unpipelined)
template <int PMODE, int QKF, bool DUMP>
__global__ __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4))) void attn_fwd(FwdArgs a) {
  constexpr bool I8 = QKF == VC_QK_INT8, F8 = QKF == VC_QK_FP8, MX = QKF == VC_QK_MXFP4;
  using SV = std::conditional_t<I8, v16i, v16f>;  // a lane's 16 scores of one 32-key block
  using QO = std::conditional_t<F8, v8i, v4i>;    // one Q or K operand of the score product
  // K_t in kb[t % 4] (MXFP4: codes, then scale bytes at MX_CODE_BYTES); V_t with its 128 bf16 block means in vb[t % 4]; mu_t / s_V as bf16 hi + lo
  // in slot t % 8 of ub[(t / 8) % 2]; (r_t, m_t) per query in slot t % 8 of rm[wave] (slot-major, so
  // that a wave's 32 queries write and read 32 consecutive 8-byte words: no bank conflicts)
  __shared__ __attribute__((aligned(16))) uint8_t kb0[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb1[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb2[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t kb3[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb0[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb1[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb2[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint8_t vb3[VBUF_BYTES];
  __shared__ __attribute__((aligned(16))) uint16_t ub[2][2][D][8];
  __shared__ __attribute__((aligned(16))) float2 rm[NW][8][32];
  __shared__ float svs[D], inv_svs[D];
  __shared__ float m_first[NW][32];  // each query's running maximum after tile 0

  // The dispatcher deals workgroups to the XCDs round-robin by linear id; the remap (a bijection
  // when the count divides evenly) gives each XCD a contiguous range of (head, query tile) pairs,
  // so its L2 serves one or two heads' K/V tiles instead of every head's (half the HBM fetches;
  // the time is unchanged, the kernel is not memory-bound)
  int qt = blockIdx.x, bh = blockIdx.y;
  {
    const int total = gridDim.x * gridDim.y, id = blockIdx.x + gridDim.x * blockIdx.y;
    if (total % NXCD == 0) {
      const int l = (id % NXCD) * (total / NXCD) + id / NXCD;
      qt = l % gridDim.x;
      bh = l / gridDim.x;
    }
  }
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kh = lane >> 5, col = lane & 31;
  const int T = a.T;
  const size_t tile0 = (size_t)bh * T;

  const int gq = NW * qt + wave;  // global 32-query group
  const int qblock = min(gq >> 2, T - 1);
  const int qrb = gq & 3;         // the group's 32-row block within its 128-row block
  // INT8: four 32-channel operands, scale sq per 128-row block; FP8: two 64-channel operands (a
  // lane holds 32 channels of its query), scale sq; MXFP4: two 64-channel operands with the E8M0
  // bytes qsc[m] of the lane's 32-channel blocks
  QO qop[I8 ? 4 : 2];
  float sq = 1.f;
  int qsc[2] = {0, 0};
  if constexpr (F8) {
    const uint8_t* qblk = reinterpret_cast<const uint8_t*>(a.q) + (tile0 + qblock) * TILE_BYTES;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const uint8_t* p = qblk + ((((qrb * 2 + m) * 2 + kh) * 2) * 32 + col) * 16;
      const u4 lo = *reinterpret_cast<const u4*>(p);
      const u4 hi = *reinterpret_cast<const u4*>(p + 512);
      qop[m] = v8i{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
    sq = a.q_scale[tile0 + qblock];
  } else if constexpr (MX) {
    const uint8_t* qblk = reinterpret_cast<const uint8_t*>(a.q) + (tile0 + qblock) * MX_CODE_BYTES;
#pragma unroll
    for (int m = 0; m < 2; ++m)
      qop[m] = *reinterpret_cast<const v4i*>(qblk + ((qrb * 2 + m) * 2 + kh) * 512 + col * 16);
    const uint2 w = *reinterpret_cast<const uint2*>(a.q_mxs + (tile0 + qblock) * MX_SCALE_BYTES + lane * 8);
    const uint32_t d = (qrb & 2) ? w.y : w.x;
#pragma unroll
    for (int m = 0; m < 2; ++m) qsc[m] = (int)((d >> (8 * ((qrb & 1) * 2 + m))) & 0xffu);
  } else {
    const int8_t* qblk = a.q + (tile0 + qblock) * TILE_BYTES;
#pragma unroll
    for (int dc = 0; dc < 4; ++dc)
      qop[dc] = *reinterpret_cast<const v4i*>(qblk + ((qrb * 4 + dc) * 2 + kh) * 512 + col * 16);
    sq = a.q_scale[tile0 + qblock];
  }

  const int mc = tid & (D - 1);
  if (tid < D) {
    const float sv = a.v_scale[(size_t)bh * D + tid];
    svs[tid] = sv;
    inv_svs[tid] = 1.f / sv;
  }
  for (int e = tid; e < 2 * 2 * D * 8 / 8; e += NTH) reinterpret_cast<u4*>(&ub[0][0][0][0])[e] = u4{0, 0, 0, 0};

  // row-sum operand of the 16x16x128 FP8 product: A rows 0 and 8 are ones on k-groups 0 and 2
  // (B lanes 0..15 and 32..47: queries 0..15), rows 4 and 12 on k-groups 1 and 3 (queries
  // 16..31); C row 4(l/16), column l%16 then holds r of query l%32 in register 0 of lane l
  v8i ones16;
  {
    const int row = lane & 15, g = lane >> 4;
    const bool on = ((row == 0 || row == 8) && !(g & 1)) || ((row == 4 || row == 12) && (g & 1));
    const int w = on ? 0x38383838 : 0;
    ones16 = v8i{w, w, w, w, w, w, w, w};
  }

  constexpr int KT_BYTES = MX ? MX_CODE_BYTES : TILE_BYTES;  // K codes per tile in memory
  const uint8_t* kbase = reinterpret_cast<const uint8_t*>(a.k) + tile0 * KT_BYTES;
  const uint8_t* ksbase = MX ? a.k_mxs + tile0 * MX_SCALE_BYTES + (MX_SCALE_BYTES / NW) * wave : nullptr;
  const uint8_t* vbase = a.v + tile0 * TILE_BYTES;
  const uint8_t* mbase = reinterpret_cast<const uint8_t*>(a.v_mean + tile0 * D) + (2 * D / NW) * wave;
  // piece u < KCOPIES of K_t into kd (every piece one copy per wave). INT8: 1 KB of codes each;
  // MXFP4: piece 0 = 1 KB of codes, piece 1 = MX_SCALE_BYTES / NW scale bytes
  auto load_kpiece = [&](int u, int t, uint8_t* kd) __attribute__((always_inline)) {
    if (!MX || u == 0) {
      const int off = (u * NW + wave) * 1024;
      copy16_to_lds(kbase + (size_t)t * KT_BYTES + off, lane * 16, lds_addr(kd + off));
    } else if (lane < MX_SCALE_BYTES / NW / 4) {
      copy4_to_lds(ksbase + (size_t)t * MX_SCALE_BYTES, 4 * lane,
                   lds_addr(kd + MX_CODE_BYTES + (MX_SCALE_BYTES / NW) * wave));
    }
  };
  auto load_k = [&](int t, uint8_t* kd) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < KCOPIES; ++u) load_kpiece(u, t, kd);
  };
  // copy k of pair p = (K_{p+2} clamped to the last tile, V_p with its means)
  auto load_part = [&](int k, int p, uint8_t* kd, uint8_t* vd) __attribute__((always_inline)) {
    if (k < KCOPIES) {
      load_kpiece(k, min(p + 2, T - 1), kd);
    } else if (k < 2 * KCOPIES) {
      const int off = ((k - KCOPIES) * NW + wave) * 1024;
      copy16_to_lds(vbase + (size_t)p * TILE_BYTES + off, lane * 16, lds_addr(vd + off));
    } else if (lane < MEAN_LANES) {
      copy4_to_lds(mbase + (size_t)p * 2 * D, 4 * lane, lds_addr(vd + TILE_BYTES + (2 * D / NW) * wave));
    }
  };
  auto load_pair = [&](int p, uint8_t* kd, uint8_t* vd) __attribute__((always_inline)) {
#pragma unroll
    for (int k = 0; k < PAIR_COPIES; ++k) load_part(k, p, kd, vd);
  };
  const __attribute__((address_space(4))) float* kscale =
      (const __attribute__((address_space(4))) float*)(MX ? nullptr : a.k_scale + tile0);
  // mu_j / s_V as bf16 hi + lo into slot j % 8 of chunk parity (j / 8) % 2, from the means behind
  // V_j in vt (threads 0..127, one channel each)
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
  SV s[4];         // scores of the tile whose codes are computed next
  v8i pc[2];       // codes of the tile whose value product is issued next
  float ksc = 0.f;  // scale of the K tile whose scores are in s
  float2* rm_q = &rm[wave][0][col];   // slot t at rm_q[32 t]

  // O^T += M^T R for the tiles of chunk parity `par` whose slot is <= last_slot, R_t = r_t 2^(m_t - m).
  // k-slots 0..7 (lanes with kh = 0) carry R_hi = bf16(R), slots 8..15 (kh = 1) R_lo = bf16(R - R_hi)
  // (R - R_hi is exact in fp32, and fma(-kh, R_hi, R) is R itself for kh = 0), against mu_hi in the
  // first product and mu_lo in the second: the four cross terms of the two splits.
  const float khf = (float)kh;
  auto flush_means = [&](int par, int last_slot) __attribute__((always_inline)) {
    float R[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float2 e = rm_q[32 * t];
      R[t] = t <= last_slot ? e.x * __builtin_amdgcn_exp2f(e.y - m_run) : 0.f;
    }
    bf16x8 b;
#pragma unroll
    for (int t = 0; t < 8; t += 2) {
      const v2f hi = __builtin_convertvector(__builtin_convertvector((v2f){R[t], R[t + 1]}, bf16x2), v2f);
      const v2f part = {__builtin_fmaf(-khf, hi[0], R[t]), __builtin_fmaf(-khf, hi[1], R[t + 1])};
      const bf16x2 v = __builtin_convertvector(part, bf16x2);
      b[t] = v[0];
      b[t + 1] = v[1];
    }
#pragma unroll
    for (int db = 0; db < 4; ++db) {
      const int c = 32 * db + col;
      const bf16x8 a_hi = *reinterpret_cast<const bf16x8*>(&ub[par][0][c][0]);
      const bf16x8 a_lo = *reinterpret_cast<const bf16x8*>(&ub[par][1][c][0]);
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_hi, b, o[db], 0, 0, 0);
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_lo, b, o[db], 0, 0, 0);
    }
  };

  // value operand n of tile vt (A operand: residual codes, 32 channels x 64 keys; n = 4 kc + db)
  auto load_vop = [&](const uint8_t* vt, int n) __attribute__((always_inline)) -> v8i {
    const int kc = n >> 2, db = n & 3;
    const int base = ((((kc * 4 + db) * 2 + kh) * 2) * 32 + col) * 16;
    const u4 lo = *reinterpret_cast<const u4*>(vt + base);
    const u4 hi = *reinterpret_cast<const u4*>(vt + base + 512);
    return v8i{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };

  // scores of tile t (K_t in kt) into s
  // MXFP4 scores of key block kb from its two operands and the lane's scale dword kb/2 of the tile
  auto qk_mx = [&](auto KBC, const v4i (&k)[2], int ksw) __attribute__((always_inline)) -> v16f {
    constexpr int kb = decltype(KBC)::value;
    v16f acc = {};
    acc = mfma_f4<(kb & 1) * 2 + 0, 0>(k[0], qop[0], acc, ksw, qsc[0]);
    acc = mfma_f4<(kb & 1) * 2 + 1, 0>(k[1], qop[1], acc, ksw, qsc[1]);
    return acc;
  };
  auto mx_kops = [&](int kb, const uint8_t* kt, v4i (&k)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < 2; ++m) k[m] = *reinterpret_cast<const v4i*>(kt + ((kb * 2 + m) * 2 + kh) * 512 + col * 16);
  };
  auto mx_scales = [&](const uint8_t* kt) __attribute__((always_inline)) -> uint2 {
    return *reinterpret_cast<const uint2*>(kt + MX_CODE_BYTES + lane * 8);
  };
  // FP8 key operands of block kb: 32 bytes per lane as two 16-byte halves 512 bytes apart
  auto f8_kops = [&](int kb, const uint8_t* kt, v8i (&k)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const uint8_t* p = kt + ((((kb * 2 + m) * 2 + kh) * 2) * 32 + col) * 16;
      const u4 lo = *reinterpret_cast<const u4*>(p);
      const u4 hi = *reinterpret_cast<const u4*>(p + 512);
      k[m] = v8i{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
  };

  // scores of tile t (K_t in kt) into s
  auto qk = [&](auto MASKC, int t, const uint8_t* kt) __attribute__((always_inline)) {
    if constexpr (MX) {
      const uint2 ksw = mx_scales(kt);
      v4i kops[2];
      mx_kops(0, kt, kops);
      s[0] = qk_mx(std::integral_constant<int, 0>{}, kops, (int)ksw.x);
      mx_kops(1, kt, kops);
      s[1] = qk_mx(std::integral_constant<int, 1>{}, kops, (int)ksw.x);
      mx_kops(2, kt, kops);
      s[2] = qk_mx(std::integral_constant<int, 2>{}, kops, (int)ksw.y);
      mx_kops(3, kt, kops);
      s[3] = qk_mx(std::integral_constant<int, 3>{}, kops, (int)ksw.y);
    } else if constexpr (F8) {
      ksc = kscale[t];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        v8i kops[2];
        f8_kops(kb, kt, kops);
        v16f acc = {};
        acc = mfma_f8(kops[0], qop[0], acc);
        s[kb] = mfma_f8(kops[1], qop[1], acc);
      }
    } else {
      ksc = kscale[t];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        v4i kops[4];
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) kops[dc] = *reinterpret_cast<const v4i*>(kt + ((kb * 4 + dc) * 2 + kh) * 512 + col * 16);
        v16i acc = {};
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) acc = mfma_i8(kops[dc], qop[dc], acc);
        s[kb] = acc;
      }
    }
    if (decltype(MASKC)::value) mask_tile(s, kh, a.N - (T - 1) * BLK);
  };

  // running maximum of tile t (scores in s) into m_new, alpha, codes into pn
  auto softmax = [&](auto LASTC, int t, v8i (&pn)[2], float& alpha, float& m_new) __attribute__((always_inline)) {
    // score scale a = fl(fl(s_q s_k) kappa) (INT8, FP8) or kappa (MXFP4: the block scales are in s)
    const float a_s = MX ? a.kappa : (sq * ksc) * a.kappa;
    using E = std::remove_reference_t<decltype(s[0][0])>;
    E mk[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      E m = smax(s[kb][0], s[kb][1]);
#pragma unroll
      for (int r = 2; r < 16; r += 2) m = smax3(m, s[kb][r], s[kb][r + 1]);
      mk[kb] = m;
    }
    E mx = smax(smax(mk[0], mk[1]), smax(mk[2], mk[3]));
    mx = half_max(mx);
    m_new = fmaxf(m_run, (float)mx * a_s);
    alpha = __builtin_amdgcn_exp2f(m_run - m_new);
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
        pn[kb >> 1][4 * (kb & 1) + d4] = (int)w;
      }
    if (PMODE == 0 && __builtin_amdgcn_ballot_w64(fabsf(m_new) >= WIDE_MAX)) clip_codes(pn);
    if (decltype(LASTC)::value) clear_padded(pn, kh, a.N - t * BLK);
  };

  const std::integral_constant<bool, false> NO;
  const std::integral_constant<bool, true> YES;

  auto pin_state = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < 4; ++db) pin(o[db]);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) pin(s[kb]);
    pin(pc[0]);
    pin(pc[1]);
    pin(l_run);
    pin(m_run);
    pin(ksc);
  };
  // codes of tile j (in pc) into row q of a.p_codes, dword w of chunk kc = keys 32(2kc + w/4) +
  // 8(w%4) + 4kh .. +3; then every copy in flight and these stores complete, which leaves the
  // copy counting of the schedule as it is
  const int q_dump = qt * NQ + wave * 32 + col;
  auto dump_codes = [&](int j) __attribute__((always_inline)) {
    if constexpr (DUMP) {
      if (q_dump < a.N) {
        uint8_t* row = a.p_codes + ((size_t)bh * a.N + q_dump) * ((size_t)T * BLK) + (size_t)j * BLK + 4 * kh;
#pragma unroll
        for (int kc = 0; kc < 2; ++kc)
#pragma unroll
          for (int w = 0; w < 8; ++w)
            *reinterpret_cast<int*>(row + 32 * (2 * kc + (w >> 2)) + 8 * (w & 3)) = pc[kc][w];
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
  };
  auto end_iter = [&](int npairs) __attribute__((always_inline)) {
    pin_state();
    wait_pairs(npairs);
    wg_barrier();
    pin_state();
  };

  // iteration j: value product and row sum of tile j (codes pc, V_j in vt); codes of tile j+1
  // (SOFTC; LASTC: it is the ragged last tile); scores of tile j+2 (QKC, K_{j+2} in kt; MASKC:
  // the last tile); pair j+3 copied into (kd, vd) (COPYC); mean j stashed; rescale to m_{j+1}
  auto iter = [&](auto COPYC, auto SOFTC, auto QKC, auto MASKC, auto LASTC, int j, const uint8_t* vt,
                  const uint8_t* kt, uint8_t* kd, uint8_t* vd) __attribute__((always_inline)) {
    constexpr bool cp = decltype(COPYC)::value, soft = decltype(SOFTC)::value, doqk = decltype(QKC)::value;
    dump_codes(j);
    v8i vop[8];
#pragma unroll
    for (int n = 0; n < 8; ++n) vop[n] = load_vop(vt, n);
    v4f rs = {};
    rs = mfma_f8_16(ones16, pc[0], rs);
    rs = mfma_f8_16(ones16, pc[1], rs);
#pragma unroll
    for (int n = 0; n < 8; ++n) {
      o[n & 3] = mfma_f8(vop[n], pc[n >> 2], o[n & 3]);
      if (cp && n < PAIR_COPIES) load_part(n, j + 3, kd, vd);
    }
    if (cp)
#pragma unroll
      for (int k = 8; k < PAIR_COPIES; ++k) load_part(k, j + 3, kd, vd);
    v8i pn[2];
    float alpha = 1.f, m_new = m_run;
    if (soft) softmax(LASTC, j + 1, pn, alpha, m_new);
    if (doqk) qk(MASKC, j + 2, kt);
    const float rsum = rs[0];
    if (a.smooth_v && j >= 8 && (j & 7) == 0) flush_means(((j >> 3) - 1) & 1, 7);
    rm_q[32 * (j & 7)] = make_float2(rsum, m_run);
    l_run += rsum;
    if (tid < D) stash_mean(j, vt);
    if (soft) {
      if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        l_run *= alpha;
      }
      m_run = m_new;
      pc[0] = pn[0];
      pc[1] = pn[1];
    }
    end_iter(cp ? 2 : 0);
  };

  // steady-state iteration j (codes of tile j+1 and scores of tile j+2 exist, neither is the last
  // tile), issued in regions that each pair matrix work with vector work of about the same
  // length; the scheduling barriers keep the regions in this order, so the scores of key block
  // kb of tile j+2 are written only after the codes of key block kb of tile j+1 are formed.
  // The wave's issue priority steps down from 3 to 0 over the regions: of the two waves sharing a
  // SIMD, the one further behind in the iteration wins the arbitration, so both reach the
  // barrier together (with equal priorities the older wave runs ahead and the other finishes the
  // iteration alone, without a partner to overlap its matrix and vector work)
  auto fence = []() __attribute__((always_inline)) { __builtin_amdgcn_sched_barrier(0); };
  auto iter_fast = [&](auto COPYC, int j, const uint8_t* vt, const uint8_t* kt, uint8_t* kd, uint8_t* vd) __attribute__((always_inline)) {
    constexpr bool cp = decltype(COPYC)::value;
    dump_codes(j);
    __builtin_amdgcn_s_setprio(3);
    auto hook = [&](int k) __attribute__((always_inline)) {
      if (cp && k < PAIR_COPIES) load_part(k, j + 3, kd, vd);
    };
    using E = std::remove_reference_t<decltype(s[0][0])>;
    auto kmax = [&](int kb) __attribute__((always_inline)) -> E {
      E m = smax(s[kb][0], s[kb][1]);
#pragma unroll
      for (int r = 2; r < 16; r += 2) m = smax3(m, s[kb][r], s[kb][r + 1]);
      return m;
    };
    // key operands of block kb (INT8: 4 x 32 channels; FP8: 2 x 64 channels; MXFP4: 2 x 64
    // channels and, with block 0, the lane's two scale dwords of the tile)
    constexpr int NKOP = I8 ? 4 : 2;
    uint2 ksw = {0u, 0u};
    auto load_kops = [&](int kb, QO (&k)[NKOP]) __attribute__((always_inline)) {
      if constexpr (MX) {
        if (kb == 0) ksw = mx_scales(kt);
        mx_kops(kb, kt, k);
      } else if constexpr (F8) {
        f8_kops(kb, kt, k);
      } else {
#pragma unroll
        for (int dc = 0; dc < 4; ++dc) k[dc] = *reinterpret_cast<const v4i*>(kt + ((kb * 4 + dc) * 2 + kh) * 512 + col * 16);
      }
    };
    auto qk_kb = [&](auto KBC, const QO (&k)[NKOP]) __attribute__((always_inline)) {
      constexpr int kb = decltype(KBC)::value;
      if constexpr (MX) {
        s[kb] = qk_mx(KBC, k, kb < 2 ? (int)ksw.x : (int)ksw.y);
      } else if constexpr (F8) {
        v16f acc = {};
        acc = mfma_f8(k[0], qop[0], acc);
        s[kb] = mfma_f8(k[1], qop[1], acc);
      } else {
        v16i acc = {};
#pragma unroll
        for (int dc = 0; dc < NKOP; ++dc) acc = mfma_i8(k[dc], qop[dc], acc);
        s[kb] = acc;
      }
    };
    v8i pn[2];
    float a8t = 0.f, bt = 0.f, a_s = 0.f, m_new = 0.f;
    // codes of key block kb. ExpCast: the fma is evaluated scaled by 2^-24, which is exact
    // (fl(2^-24 x) = 2^-24 fl(x)), with the clamp at 0 folded into it; below 2^-13 the fp16 spacing
    // is 2^-24, so the fp16 conversion of each pair rounds to the nearest-even integer code and
    // leaves it in the low bits, and one byte permute packs four (codes below 256: see WIDE_MAX)
    auto codes_kb = [&](int kb) __attribute__((always_inline)) {
#pragma unroll
      for (int d4 = 0; d4 < 4; ++d4) {
        uint32_t w = 0;
        if (PMODE == 0) {
          float z[4];
#pragma unroll
          for (int q = 0; q < 4; ++q)
            z[q] = __builtin_amdgcn_fmed3f(__builtin_fmaf((float)s[kb][4 * d4 + q], a8t, bt), 0.f, 1.f);
          const h2 lo = __builtin_convertvector((v2f){z[0], z[1]}, h2);
          const h2 hi = __builtin_convertvector((v2f){z[2], z[3]}, h2);
          w = __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, hi), __builtin_bit_cast(uint32_t, lo), 0x06040200u);
        } else {
          float pe[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) pe[q] = __builtin_amdgcn_exp2f((float)s[kb][4 * d4 + q] * a_s - m_new) * 256.f;
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(pe[0], pe[1], 0, false);
          w = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(pe[2], pe[3], (int)w, true);
        }
        int wi = (int)w;
        pin(wi);  // formed in this region (pure values would otherwise be placed next to their use)
        pn[kb >> 1][4 * (kb & 1) + d4] = wi;
      }
    };
    // at most 32 registers of operands staged at any time
    v8i va[2], vb[2];
    QO k0[NKOP], k1[NKOP];
    // R0: value operands 0, 1
    va[0] = load_vop(vt, 0);
    va[1] = load_vop(vt, 1);
    hook(0);
    fence();
    // R1: row sum and value products 0, 1; operands 2, 3; maxima of key blocks 0, 1
    v4f rs = mfma_f8_16(ones16, pc[0], v4f{});
    o[0] = mfma_f8(va[0], pc[0], o[0]);
    o[1] = mfma_f8(va[1], pc[0], o[1]);
    vb[0] = load_vop(vt, 2);
    vb[1] = load_vop(vt, 3);
    E mk0 = kmax(0), mk1 = kmax(1);
    pin(mk0);
    pin(mk1);
    fence();
    __builtin_amdgcn_s_setprio(2);
    fence();
    // R2: value products 2, 3; operands 4, 5; maxima of blocks 2, 3, m', alpha
    o[2] = mfma_f8(vb[0], pc[0], o[2]);
    o[3] = mfma_f8(vb[1], pc[0], o[3]);
    va[0] = load_vop(vt, 4);
    va[1] = load_vop(vt, 5);
    a_s = MX ? a.kappa : (sq * ksc) * a.kappa;  // fl(fl(s_q s_k) kappa) for INT8 and FP8
    E mx = smax(smax(mk0, mk1), smax(kmax(2), kmax(3)));
    mx = half_max(mx);
    m_new = fmaxf(m_run, (float)mx * a_s);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float alpha_p = alpha;
    a8t = a_s * 0x1p-21f;                                       // 2^-24 8a
    bt = __builtin_fmaf(m_new, -0x1p-21f, a.cbias * 0x1p-24f);  // 2^-24 fl(cbias - 8m')
    pin(alpha_p);
    pin(a8t);
    pin(bt);
    pin(m_new);
    const bool wide = PMODE == 0 && __builtin_amdgcn_ballot_w64(fabsf(m_new) >= WIDE_MAX);
    hook(1);
    fence();
    // R3: row sum and value products 4, 5; operands 6, 7; key operands of block 0; codes of block 0
    rs = mfma_f8_16(ones16, pc[1], rs);
    o[0] = mfma_f8(va[0], pc[1], o[0]);
    o[1] = mfma_f8(va[1], pc[1], o[1]);
    vb[0] = load_vop(vt, 6);
    vb[1] = load_vop(vt, 7);
    codes_kb(0);
    hook(2);
    fence();
    __builtin_amdgcn_s_setprio(1);
    fence();
    // R4: value products 6, 7, scores of block 0; key operands of block 1; codes of block 1
    load_kops(0, k0);
    o[2] = mfma_f8(vb[0], pc[1], o[2]);
    o[3] = mfma_f8(vb[1], pc[1], o[3]);
    qk_kb(std::integral_constant<int, 0>{}, k0);
    codes_kb(1);
    hook(3);
    fence();
    // R5: scores of block 1; key operands of block 2; codes of block 2
    load_kops(1, k1);
    qk_kb(std::integral_constant<int, 1>{}, k1);
    load_kops(2, k0);
    codes_kb(2);
    hook(4);
    fence();
    __builtin_amdgcn_s_setprio(0);
    fence();
    // R6: scores of block 2; key operands of block 3; codes of block 3
    qk_kb(std::integral_constant<int, 2>{}, k0);
    load_kops(3, k1);
    codes_kb(3);
    fence();
    // R7: scores of block 3
    qk_kb(std::integral_constant<int, 3>{}, k1);
    if (!MX) ksc = kscale[j + 2];
    const float rsum = rs[0];
    if (a.smooth_v && j >= 8 && (j & 7) == 0) flush_means(((j >> 3) - 1) & 1, 7);
    rm_q[32 * (j & 7)] = make_float2(rsum, m_run);
    l_run += rsum;
    if (tid < D) stash_mean(j, vt);
    if (__builtin_amdgcn_ballot_w64(alpha_p != 1.f)) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha_p;
      l_run *= alpha_p;
    }
    m_run = m_new;
    if (wide) clip_codes(pn);
    pc[0] = pn[0];
    pc[1] = pn[1];
    end_iter(cp ? 2 : 0);
  };

  // prologue: K_0, K_1, pairs 0 and 1; scores of tile 0, its codes, scores of tile 1; pair 2
  const bool t2 = T > 1, t3 = T > 2;
  wait_pairs(0);  // the compiler's own loads have landed before any copy
  load_k(0, kb0);
  if (t2) load_k(1, kb1);
  load_pair(0, kb2, vb0);
  if (t2) load_pair(1, kb3, vb1);
  wait_pairs(t2 ? 2 : 1);  // K_0, K_1
  wg_barrier();
  if (T == 1) qk(YES, 0, kb0);
  else qk(NO, 0, kb0);
  {
    float alpha, m_new;
    if (T == 1) softmax(YES, 0, pc, alpha, m_new);
    else softmax(NO, 0, pc, alpha, m_new);
    m_run = m_new;
    if (kh == 0) m_first[wave][col] = m_run;
  }
  if (t2) {
    if (T == 2) qk(YES, 1, kb1);
    else qk(NO, 1, kb1);
  }
  pin_state();
  wg_barrier();  // every wave is done with K_0 before pair 2 overwrites it
  if (t3) load_pair(2, kb0, vb2);
  end_iter((int)t2 + (int)t3);  // pair 0

  // steady state (pair j+3 exists), unrolled by four so every buffer is named statically:
  // V_j in vb[j%4], K_{j+2} in kb[(j+2)%4], pair j+3 into (kb[(j+1)%4], vb[(j+3)%4])
  int j = 0;
  for (; j + 6 <= T - 1; j += 4) {  // the group's last iteration j + 3 still copies pair j + 6
    iter_fast(YES, j, vb0, kb2, kb1, vb3);
    iter_fast(YES, j + 1, vb1, kb3, kb2, vb0);
    iter_fast(YES, j + 2, vb2, kb0, kb3, vb1);
    iter_fast(YES, j + 3, vb3, kb1, kb0, vb2);
  }
  if (j + 3 <= T - 1) {
    iter_fast(YES, j, vb0, kb2, kb1, vb3);
    ++j;
    if (j + 3 <= T - 1) {
      iter_fast(YES, j, vb1, kb3, kb2, vb0);
      ++j;
      if (j + 3 <= T - 1) {
        iter_fast(YES, j, vb2, kb0, kb3, vb1);
        ++j;
      }
    }
  }
  __builtin_amdgcn_s_setprio(0);
  auto kbuf = [&](int b) __attribute__((always_inline)) -> const uint8_t* {
    return b == 0 ? kb0 : (b == 1 ? kb1 : (b == 2 ? kb2 : kb3));
  };
  auto vbuf = [&](int b) __attribute__((always_inline)) -> const uint8_t* {
    return b == 0 ? vb0 : (b == 1 ? vb1 : (b == 2 ? vb2 : vb3));
  };
  // tail: iterations T-3 (scores of the last tile), T-2 (codes of the last tile), T-1
  if (j == T - 3) {
    iter(NO, YES, YES, YES, NO, j, vbuf(j & 3), kbuf((j + 2) & 3), kb0, vb0);
    ++j;
  }
  if (j == T - 2) {
    iter(NO, YES, NO, NO, YES, j, vbuf(j & 3), kb0, kb0, vb0);
    ++j;
  }
  iter(NO, NO, NO, NO, NO, T - 1, vbuf((T - 1) & 3), kb0, kb0, vb0);
  if (a.smooth_v) flush_means(((T - 1) >> 3) & 1, (T - 1) & 7);

  // epilogue: O = A s_V / l, bf16, row q written to token q_perm[q] (or q)
  const int q = qt * NQ + wave * 32 + col;
  if (q < a.N) {
    // a row outside the domain of the fp16 code conversion is written as NaN
    const bool out_of_domain = PMODE == 0 && (fabsf(m_first[wave][col]) >= DOMAIN_MAX || fabsf(m_run) >= DOMAIN_MAX);
    const float inv_l = out_of_domain ? __builtin_nanf("") : 1.f / l_run;
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

// The FP8 score product on caller data (vc_fp8_score_product): one wave per 32x32 block, the two
// chained 32x32x64 instructions of the scores of a 32-key block (A = rows of a, B = rows of b),
// from the accumulator c_in. Operand lane l holds row l % 32, channels 64m + 32(l / 32) .. + 31.
__global__ __launch_bounds__(64) void fp8_score_product(const uint8_t* a, const uint8_t* b, const float* c_in,
                                                        float* out) {
  const int lane = threadIdx.x, row = lane & 31, half = lane >> 5;
  const size_t blk = blockIdx.x;
  const uint8_t* ar = a + (blk * 32 + row) * D + 32 * half;
  const uint8_t* br = b + (blk * 32 + row) * D + 32 * half;
  auto op = [](const uint8_t* p) -> v8i {
    const u4 lo = *reinterpret_cast<const u4*>(p), hi = *reinterpret_cast<const u4*>(p + 16);
    return v8i{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3], (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  };
  // C register r of lane l: row 8(r/4) + 4(l/32) + r%4, column l%32
  v16f acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = c_in[(blk * 32 + 8 * (r >> 2) + 4 * half + (r & 3)) * 32 + row];
  acc = mfma_f8(op(ar), op(br), acc);
  acc = mfma_f8(op(ar + 64), op(br + 64), acc);
#pragma unroll
  for (int r = 0; r < 16; ++r) out[(blk * 32 + 8 * (r >> 2) + 4 * half + (r & 3)) * 32 + row] = acc[r];
}

hipError_t launch_fp8_score_product(const uint8_t* a, const uint8_t* b, const float* c_in, float* out, int n,
                                    hipStream_t s) {
  fp8_score_product<<<n, 64, 0, s>>>(a, b, c_in, out);
  return hipGetLastError();
}

hipError_t launch_forward(const FwdArgs& a, int BH, hipStream_t s) {
  const dim3 grid((a.N + NQ - 1) / NQ, BH);
  auto go = [&](auto PC, auto DC) {
    constexpr int pm = decltype(PC)::value;
    constexpr bool dump = decltype(DC)::value;
    if (a.qk_fmt == VC_QK_MXFP4) attn_fwd<pm, VC_QK_MXFP4, dump><<<grid, NTH, 0, s>>>(a);
    else if (a.qk_fmt == VC_QK_FP8) attn_fwd<pm, VC_QK_FP8, dump><<<grid, NTH, 0, s>>>(a);
    else attn_fwd<pm, VC_QK_INT8, dump><<<grid, NTH, 0, s>>>(a);
  };
  const std::integral_constant<int, 0> EXPCAST;
  const std::integral_constant<int, 1> EXPTHENCAST;
  const std::integral_constant<bool, true> DUMP;
  const std::integral_constant<bool, false> NODUMP;
  if (a.p_codes) {
    if (a.p_mode == 0) go(EXPCAST, DUMP);
    else go(EXPTHENCAST, DUMP);
  } else {
    if (a.p_mode == 0) go(EXPCAST, NODUMP);
    else go(EXPTHENCAST, NODUMP);
  }
  return hipGetLastError();
}

}  // namespace vc
