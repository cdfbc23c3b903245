// Internal launch arguments and launchers (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vc_attn.h"

namespace vc {

struct PrepArgs {
  const uint16_t *Q, *K, *V;
  const int32_t *perm, *q_perm;
  const float *rope_cos, *rope_sin;
  int8_t* q;
  float* q_scale;
  int8_t* k;
  float* k_scale;
  float* k_mean;
  uint8_t* v;
  float* v_scale;
  uint16_t* v_mean;
  uint8_t *q_mxs, *k_mxs;  // E8M0 scale bytes (MXFP4 only)
  float* ws_ksum;   // [B*H][T][128] per-block key channel sums
  float* ws_vamax;  // [B*H][T][128] per-block residual maxima
  float* ws_vinv;   // [B*H][128]    448 / amax (0 for an all-zero channel)
  int N, T, F, Ht, Wd;
  float inv_w, inv_hw;  // 1/Wd and 1/(Ht*Wd) in fp32: estimates for the token-position divisions
  int rope, hadamard, smooth_k, smooth_v;
  int qk_fmt;
};

struct FwdArgs {
  const int8_t* q;
  const float* q_scale;
  const int8_t* k;
  const float* k_scale;
  const uint8_t* v;
  const float* v_scale;
  const uint16_t* v_mean;
  const uint8_t *q_mxs, *k_mxs;  // E8M0 scale bytes (MXFP4 only)
  const int32_t* q_perm;
  uint16_t* O;
  uint8_t* p_codes;  // debugging: the probability codes of every tile [B*H][N][128 T], or null
  int N, T;
  float kappa;      // sm_scale * log2(e) (/ 128 with the Hadamard rotation), rounded once to fp32
  float cbias;      // fl(120 + beta)
  int p_mode, smooth_v;
  int qk_fmt;
};

struct GroupArgs {
  const uint16_t* V;
  float* centroids;
  int32_t *labels, *perm, *inv_perm;
  int8_t* codes;     // workspace: per-head INT8 codes of V [B*H][N][128]
  float* scale;      // workspace: [B*H] amax (then scale)
  int32_t* cent;     // workspace: [B*H][k][128] integer centroids
  int8_t* cent8;     // workspace: [B*H][64][128] the same as int8, rows k.. zero
  int32_t* cnorm;    // workspace: [B*H][64] their squared norms, rows k.. a padding value
  int32_t* sums;     // workspace: [B*H][npart][k][128] member sums per assignment workgroup
  int32_t* counts;   // workspace: [B*H][npart][k] member counts, later [B*H][nblk][k] label histograms
  int32_t* blockhist;// workspace: [B*H][nblk][nlab] per-block label counts, then offsets
  int N, F, Ht, Wd, k, iters, warm_start, mode, cube_t, cube_h, cube_w, nlab, nblk;
  int npart;         // assignment workgroups per head (1024 tokens each)
};

hipError_t launch_prep(const PrepArgs& a, int BH, hipStream_t s);
hipError_t launch_forward(const FwdArgs& a, int BH, hipStream_t s);
hipError_t launch_group(const GroupArgs& a, int BH, hipStream_t s);
hipError_t launch_fp8_score_product(const uint8_t* a, const uint8_t* b, const float* c_in, float* out, int n,
                                    hipStream_t s);

}  // namespace vc
