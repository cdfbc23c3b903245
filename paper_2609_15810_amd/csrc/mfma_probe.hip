// Matrix-core limits of this GPU that bound the attention kernel, measured rather than taken from
// the data sheet. Standalone program (no library code), printed as one JSON object.
//
// 1. Sustained rate and core clock of the products the attention kernel is built from, INT8
//    32x32x32 (scores), FP8 32x32x64 (value products) and, for the 4-bit variant's scores, the
//    scaled FP4 32x32x64 (E2M1 operands, unit E8M0 scales), four independent accumulator chains per
//    wave, two waves per SIMD, every CU busy. Operands either constant or random bytes (xorshift
//    per lane; FP8 bytes masked with 0x77 so no NaN encodings occur). The clock is the ratio of the
//    shader clock counter (s_memtime) to the 100 MHz constant counter (s_memrealtime) over each
//    workgroup's lifetime. With random operands the chip lowers its clock to stay in its power
//    budget, so these rates are the ceiling a product on real data can reach.
// 2. How much vector work one wave issues under its own product: one wave per SIMD runs groups of
//    one product followed by n independent v_fma_f32; the cycles per group against the product's
//    own cycles + 4 n (a wave64 VALU instruction takes 4 cycles) give the overlapped cycles.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

#define CHECK(x)                                                                  \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));         \
      std::exit(1);                                                               \
    }                                                                             \
  } while (0)

__device__ __forceinline__ v16i mm_i8(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mm_f8(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}
// FP4 x FP4 (cbsz = blgp = 4: 32 E2M1 codes in the low four registers), E8M0 scales 127 (= 1)
__device__ __forceinline__ v16f mm_f4(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 4, 4, 0, 127, 0, 127);
}

// Part 1. KIND 0: INT8 32x32x32, 1: FP8 32x32x64, 2: FP4 32x32x64; RND: random operands (else
// constant ones; every E2M1 code is finite, so FP4 takes any byte). Each workgroup writes its lane
// sums to out[block * blockDim + thread] (so nothing is removed as dead) and, from thread 0, its
// shader-clock and constant-clock spans to clk[2 block .. + 1].
template <int KIND, bool RND>
__global__ __launch_bounds__(512) void rate(int iters, float* out, unsigned long long* clk) {
  constexpr bool F8 = KIND == 1;
  const int l = threadIdx.x;
  const unsigned long long t0 = __builtin_readcyclecounter();
  const unsigned long long w0 = __builtin_amdgcn_s_memrealtime();
  unsigned x = 2654435761u * (unsigned)(l + 1) + 97u * blockIdx.x;
  auto word = [&]() -> int {
    if (!RND) return 0x3a3a3a3a;  // FP8 0.75 / INT8 58 in every byte
    x ^= x << 13;
    x ^= x >> 17;
    x ^= x << 5;
    return (int)(F8 ? (x & 0x77777777u) : x);
  };
  v8i r[4];
  for (int m = 0; m < 4; ++m) r[m] = v8i{word(), word(), word(), word(), word(), word(), word(), word()};
  float sum = 0.f;
  if constexpr (KIND == 1 || KIND == 2) {
    auto mm = [](v8i a, v8i b, v16f c) { return KIND == 1 ? mm_f8(a, b, c) : mm_f4(a, b, c); };
    v16f c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int i = 0; i < iters; ++i) {
      c0 = mm(r[0], r[1], c0);
      c1 = mm(r[2], r[3], c1);
      c2 = mm(r[1], r[2], c2);
      c3 = mm(r[3], r[0], c3);
    }
    for (int q = 0; q < 16; ++q) sum += c0[q] + c1[q] + c2[q] + c3[q];
  } else {
    auto lo = [](v8i v) { return v4i{v[0], v[1], v[2], v[3]}; };
    auto hi = [](v8i v) { return v4i{v[4], v[5], v[6], v[7]}; };
    v16i c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int i = 0; i < iters; ++i) {
      c0 = mm_i8(lo(r[0]), hi(r[1]), c0);
      c1 = mm_i8(lo(r[2]), hi(r[3]), c1);
      c2 = mm_i8(hi(r[0]), lo(r[3]), c2);
      c3 = mm_i8(hi(r[2]), lo(r[1]), c3);
    }
    for (int q = 0; q < 16; ++q) sum += (float)(c0[q] + c1[q] + c2[q] + c3[q]);
  }
  const unsigned long long t1 = __builtin_readcyclecounter();
  const unsigned long long w1 = __builtin_amdgcn_s_memrealtime();
  out[(size_t)blockIdx.x * blockDim.x + l] = sum;
  if (l == 0) {
    clk[2 * blockIdx.x] = t1 - t0;
    clk[2 * blockIdx.x + 1] = w1 - w0;
  }
}

// Part 2. One product (accumulators alternating between two chains) then NV independent v_fma_f32
// on four private registers, in that order (the scheduling barrier keeps each group together).
// Thread 0 of each workgroup writes its shader-clock span to clk[block].
template <bool F8, int NV>
__global__ __launch_bounds__(256) void cover(int iters, float* out, unsigned long long* clk) {
  const int l = threadIdx.x;
  const v4i a4 = {l, l + 1, l + 2, l + 3};
  const v8i a8 = {l & 0x37, l & 0x35, l & 0x33, l & 0x31, l & 0x27, l & 0x25, l & 0x23, l & 0x21};
  float x0 = (float)l, x1 = x0 + 1.f, x2 = x0 + 2.f, x3 = x0 + 3.f;
  const float y = 1.0001f, z = 0.5f;
  v16i c0 = {}, c1 = {};
  v16f d0 = {}, d1 = {};
  const unsigned long long t0 = __builtin_readcyclecounter();
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      if constexpr (F8) {
        if (g & 1) d1 = mm_f8(a8, a8, d1);
        else d0 = mm_f8(a8, a8, d0);
      } else {
        if (g & 1) c1 = mm_i8(a4, a4, c1);
        else c0 = mm_i8(a4, a4, c0);
      }
#pragma unroll
      for (int k = 0; k < NV / 4; ++k) {
        asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(x0) : "v"(y), "v"(z));
        asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(x1) : "v"(y), "v"(z));
        asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(x2) : "v"(y), "v"(z));
        asm volatile("v_fma_f32 %0, %0, %1, %2" : "+v"(x3) : "v"(y), "v"(z));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const unsigned long long t1 = __builtin_readcyclecounter();
  float s = x0 + x1 + x2 + x3;
  for (int q = 0; q < 16; ++q) s += (float)(c0[q] + c1[q]) + d0[q] + d1[q];
  out[(size_t)blockIdx.x * blockDim.x + l] = s;
  if (l == 0) clk[blockIdx.x] = t1 - t0;
}

int main() {
  int ncu = 0;
  CHECK(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, 0));
  const int nblk = 8 * ncu;  // 8 workgroups of 8 waves per CU
  float* out = nullptr;
  unsigned long long* clk = nullptr;
  CHECK(hipMalloc(&out, sizeof(float) * (size_t)nblk * 512));
  CHECK(hipMalloc(&clk, sizeof(unsigned long long) * 2 * (size_t)nblk));
  std::vector<unsigned long long> h(2 * (size_t)nblk);
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));

  std::printf("{\"cus\": %d, \"rate\": {", ncu);
  struct Case { const char* name; int kind; bool rnd; double ops; int iters; };
  const Case cases[6] = {{"int8_32x32x32_constant", 0, false, 32.0 * 32 * 32 * 2, 4000},
                         {"int8_32x32x32_random", 0, true, 32.0 * 32 * 32 * 2, 4000},
                         {"fp8_32x32x64_constant", 1, false, 32.0 * 32 * 64 * 2, 2000},
                         {"fp8_32x32x64_random", 1, true, 32.0 * 32 * 64 * 2, 2000},
                         {"fp4_32x32x64_constant", 2, false, 32.0 * 32 * 64 * 2, 4000},
                         {"fp4_32x32x64_random", 2, true, 32.0 * 32 * 64 * 2, 4000}};
  for (int c = 0; c < 6; ++c) {
    const int iters = cases[c].iters;
    auto launch = [&]() {
      switch (c) {
        case 0: rate<0, false><<<nblk, 512>>>(iters, out, clk); break;
        case 1: rate<0, true><<<nblk, 512>>>(iters, out, clk); break;
        case 2: rate<1, false><<<nblk, 512>>>(iters, out, clk); break;
        case 3: rate<1, true><<<nblk, 512>>>(iters, out, clk); break;
        case 4: rate<2, false><<<nblk, 512>>>(iters, out, clk); break;
        default: rate<2, true><<<nblk, 512>>>(iters, out, clk); break;
      }
    };
    float ms = 0.f;
    for (int rep = 0; rep < 4; ++rep) {  // the clock settles over the first launches; the last counts
      CHECK(hipEventRecord(e0));
      launch();
      CHECK(hipEventRecord(e1));
      CHECK(hipEventSynchronize(e1));
      CHECK(hipGetLastError());
    }
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    CHECK(hipMemcpy(h.data(), clk, sizeof(unsigned long long) * 2 * nblk, hipMemcpyDeviceToHost));
    double cyc = 0, ticks = 0;
    for (int b = 0; b < nblk; ++b) {
      cyc += (double)h[2 * b];
      ticks += (double)h[2 * b + 1];
    }
    const double ops = cases[c].ops * 4.0 * iters * 8.0 * nblk;  // 4 chains, 8 waves per workgroup
    std::printf("%s\"%s\": {\"tops\": %.1f, \"clock_ghz\": %.3f, \"ms\": %.3f}", c ? ", " : "", cases[c].name,
                ops / (ms * 1e-3) / 1e12, cyc / (ticks / 100e6) / 1e9, ms);
  }
  std::printf("}, \"cover\": {");
  struct Cov { const char* name; bool f8; int nv; int mcyc; };
  const Cov cov[6] = {{"int8_n0", false, 0, 32}, {"int8_n4", false, 4, 32}, {"int8_n8", false, 8, 32},
                      {"fp8_n0", true, 0, 64},   {"fp8_n8", true, 8, 64},   {"fp8_n16", true, 16, 64}};
  for (int c = 0; c < 6; ++c) {
    const int iters = 2000;
    auto launch = [&]() {
      switch (c) {
        case 0: cover<false, 0><<<ncu, 256>>>(iters, out, clk); break;
        case 1: cover<false, 4><<<ncu, 256>>>(iters, out, clk); break;
        case 2: cover<false, 8><<<ncu, 256>>>(iters, out, clk); break;
        case 3: cover<true, 0><<<ncu, 256>>>(iters, out, clk); break;
        case 4: cover<true, 8><<<ncu, 256>>>(iters, out, clk); break;
        default: cover<true, 16><<<ncu, 256>>>(iters, out, clk); break;
      }
    };
    for (int rep = 0; rep < 2; ++rep) {
      launch();
      CHECK(hipDeviceSynchronize());
      CHECK(hipGetLastError());
    }
    CHECK(hipMemcpy(h.data(), clk, sizeof(unsigned long long) * ncu, hipMemcpyDeviceToHost));
    double cyc = 0;
    for (int b = 0; b < ncu; ++b) cyc += (double)h[b];
    const double per = cyc / ncu / (4.0 * iters);
    const double hidden = cov[c].mcyc + 4.0 * cov[c].nv - per;
    std::printf("%s\"%s\": {\"cycles_per_group\": %.1f, \"overlapped_cycles\": %.1f}", c ? ", " : "", cov[c].name,
                per, hidden);
  }
  std::printf("}}\n");
  CHECK(hipFree(out));
  CHECK(hipFree(clk));
  return 0;
}
