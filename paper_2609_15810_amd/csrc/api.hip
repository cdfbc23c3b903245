// C ABI of the library (declared in include/vc_attn.h): argument validation on the host, the
// workspace carve-up, and the launches of the preprocessing, grouping and attention kernels.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "vc_attn.h"
#include "vc_internal.hpp"

namespace {

thread_local int g_last_hip = 0;

constexpr int kD = 128;
constexpr int kKMax = 64;

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline int blocks_of(int n, int b) { return (n + b - 1) / b; }

vc_status check_shape(const vc_shape* s) {
  if (!s) return VC_ERR_NULL;
  if (s->d != kD || s->B < 1 || s->H < 1 || s->N < 1 || s->F < 1 || s->Ht < 1 || s->Wd < 1) return VC_ERR_SHAPE;
  // F * Ht <= N < 2^31 before the last factor, so the product cannot overflow
  const long long fh = (long long)s->F * s->Ht;
  if (fh > s->N || fh * s->Wd != s->N) return VC_ERR_SHAPE;
  const long long T = blocks_of(s->N, 128);
  if ((long long)s->B * s->H * T * 128 * kD >= (1LL << 31)) return VC_ERR_SHAPE;
  return VC_OK;
}

vc_status check_opts(const vc_opts* o) {
  if (!o) return VC_ERR_NULL;
  if (o->qk_fmt != VC_QK_INT8 && o->qk_fmt != VC_QK_FP8 && o->qk_fmt != VC_QK_MXFP4) return VC_ERR_UNSUPPORTED;
  if (o->p_mode != VC_P_EXPCAST && o->p_mode != VC_P_EXP_THEN_CAST) return VC_ERR_UNSUPPORTED;
  const int32_t flags[4] = {o->rope, o->hadamard, o->smooth_k, o->smooth_v};
  for (int32_t f : flags)
    if (f != 0 && f != 1) return VC_ERR_UNSUPPORTED;
  // the score scale sm_scale * log2(e) must be finite in fp32 (NaN fails)
  if (!(o->sm_scale >= 0.f) || !std::isfinite(o->sm_scale * 1.4426950408889634f)) return VC_ERR_UNSUPPORTED;
  // -1 <= beta <= 0 (NaN fails): the row maximum's ExpCast code stays in [119, 120]
  if (!(o->beta >= -1.f && o->beta <= 0.f)) return VC_ERR_UNSUPPORTED;
  return VC_OK;
}

vc_status check_group_opts(const vc_shape* s, const vc_group_opts* g) {
  if (!g) return VC_ERR_NULL;
  if (g->mode == VC_GROUP_IDENTITY) return VC_OK;
  if (g->mode == VC_GROUP_CUBE) {
    if (g->cube[0] < 1 || g->cube[1] < 1 || g->cube[2] < 1) return VC_ERR_UNSUPPORTED;
    return VC_OK;
  }
  if (g->mode != VC_GROUP_KMEANS) return VC_ERR_UNSUPPORTED;
  if (g->k < 1 || g->k > kKMax || g->k > s->N) return VC_ERR_UNSUPPORTED;
  if (g->iters < 0 || g->iters > 64 || (g->warm_start != 0 && g->warm_start != 1)) return VC_ERR_UNSUPPORTED;
  return VC_OK;
}

size_t prep_ws(const vc_shape* s) {
  const size_t BH = (size_t)s->B * s->H, T = blocks_of(s->N, 128);
  return 2 * align256(BH * T * kD * 4) + align256(BH * kD * 4);
}

size_t group_ws(const vc_shape* s, const vc_group_opts* g) {
  if (g->mode != VC_GROUP_KMEANS) return 0;
  const size_t BH = (size_t)s->B * s->H, N = s->N, K = g->k, nblk = blocks_of(s->N, 256);
  return align256(BH * N * kD) + align256(BH * 4) + align256(BH * K * kD * 4) + align256(BH * nblk * K * kD * 4) +
         2 * align256(BH * nblk * K * 4) + align256(BH * 64 * kD) +
         align256(BH * 64 * 4);
}

vc_status hip_status(hipError_t e) {
  if (e == hipSuccess) return VC_OK;
  g_last_hip = (int)e;
  return VC_ERR_HIP;
}

// Preprocessing workspace of vc_attn_prep_noalloc: one copy per GPU, held until the process ends.
// In host code the name `scratch` is only a stand-in for the symbol; the device address of this
// GPU's copy comes from hipGetSymbolAddress, once per device, and only that address is used.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mu;

// Device address of the current GPU's scratch (looked up on the first call on that GPU).
vc_status scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (dev < 0 || dev >= kMaxDevices) return VC_ERR_INTERNAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e);
    if (!p) return VC_ERR_INTERNAL;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return VC_OK;
}

}  // namespace

extern "C" {

void vc_opts_default(vc_opts* o) {
  if (!o) return;
  o->qk_fmt = VC_QK_INT8;
  o->p_mode = VC_P_EXPCAST;
  o->rope = o->hadamard = o->smooth_k = o->smooth_v = 1;
  o->sm_scale = 0.f;
  o->beta = -0.35f;
}

void vc_group_opts_default(vc_group_opts* g) {
  if (!g) return;
  g->mode = VC_GROUP_KMEANS;
  g->k = 32;
  g->iters = 8;
  g->warm_start = 0;
  g->cube[0] = 4;
  g->cube[1] = 2;
  g->cube[2] = 16;
}

size_t vc_attn_workspace_size(const vc_shape* shape, const vc_opts* opts, const vc_group_opts* gopts) {
  if (check_shape(shape) != VC_OK) return 0;
  size_t ws = 0;
  if (opts) {
    if (check_opts(opts) != VC_OK) return 0;
    ws = prep_ws(shape);
  }
  if (gopts) {
    if (check_group_opts(shape, gopts) != VC_OK) return 0;
    const size_t g = group_ws(shape, gopts);
    ws = ws > g ? ws : g;
  }
  return ws;
}

vc_status vc_rope_tables(int32_t F, int32_t Ht, int32_t Wd, double theta, float* cos_t, float* sin_t) {
  if (!cos_t || !sin_t) return VC_ERR_NULL;
  if (F < 1 || Ht < 1 || Wd < 1 || !(theta > 0.0) || !std::isfinite(theta)) return VC_ERR_SHAPE;
  // the tables hold (F + Ht + Wd) x 64 entries each: refuse sizes whose entry count overflows int
  if ((long long)F + Ht + Wd > (1LL << 31) / 64 - 1) return VC_ERR_SHAPE;
  const int rows = F + Ht + Wd;
  for (int r = 0; r < rows; ++r) {
    const int axis = r < F ? 0 : (r < F + Ht ? 1 : 2);
    const int pos = axis == 0 ? r : (axis == 1 ? r - F : r - F - Ht);
    const int first = axis == 0 ? 0 : (axis == 1 ? 22 : 43);
    const int npair = axis == 0 ? 22 : 21;
    const double dims = axis == 0 ? 44.0 : 42.0;
    for (int i = 0; i < 64; ++i) {
      const int j = i - first;
      if (j < 0 || j >= npair) {
        cos_t[r * 64 + i] = 1.0f;
        sin_t[r * 64 + i] = 0.0f;
        continue;
      }
      const double ang = (double)pos * std::pow(theta, -(2.0 * j) / dims);
      cos_t[r * 64 + i] = (float)std::cos(ang);
      sin_t[r * 64 + i] = (float)std::sin(ang);
    }
  }
  return VC_OK;
}

vc_status vc_attn_group(const vc_shape* shape, const vc_group_opts* gopts, const uint16_t* V, float* centroids,
                        int32_t* labels, int32_t* perm, int32_t* inv_perm, void* ws, size_t ws_bytes, void* stream) {
  vc_status st = check_shape(shape);
  if (st != VC_OK) return st;
  if ((st = check_group_opts(shape, gopts)) != VC_OK) return st;
  if (!labels || !perm) return VC_ERR_NULL;
  const bool km = gopts->mode == VC_GROUP_KMEANS;
  if (km && (!V || !centroids)) return VC_ERR_NULL;
  const size_t need = group_ws(shape, gopts);
  if (need > 0 && (!ws || ws_bytes < need)) return VC_ERR_WORKSPACE;
  if ((V && !aligned16(V)) || !aligned16(labels) || !aligned16(perm) || (inv_perm && !aligned16(inv_perm)) ||
      (centroids && !aligned16(centroids)) || (ws && !aligned16(ws)))
    return VC_ERR_ALIGN;

  vc::GroupArgs a{};
  const size_t BH = (size_t)shape->B * shape->H;
  a.V = V;
  a.centroids = centroids;
  a.labels = labels;
  a.perm = perm;
  a.inv_perm = inv_perm;
  a.N = shape->N;
  a.F = shape->F;
  a.Ht = shape->Ht;
  a.Wd = shape->Wd;
  a.mode = gopts->mode;
  a.k = km ? gopts->k : 1;
  a.iters = gopts->iters;
  a.warm_start = gopts->warm_start;
  a.cube_t = gopts->cube[0];
  a.cube_h = gopts->cube[1];
  a.cube_w = gopts->cube[2];
  a.nblk = blocks_of(shape->N, 256);
  a.npart = blocks_of(shape->N, 1024);
  a.nlab = a.k;
  if (km) {
    char* p = static_cast<char*>(ws);
    const size_t N = shape->N, K = a.k, nblk = a.nblk;
    a.codes = reinterpret_cast<int8_t*>(p);
    p += align256(BH * N * kD);
    a.scale = reinterpret_cast<float*>(p);
    p += align256(BH * 4);
    a.cent = reinterpret_cast<int32_t*>(p);
    p += align256(BH * K * kD * 4);
    a.sums = reinterpret_cast<int32_t*>(p);
    p += align256(BH * nblk * K * kD * 4);
    a.counts = reinterpret_cast<int32_t*>(p);
    p += align256(BH * nblk * K * 4);
    a.blockhist = reinterpret_cast<int32_t*>(p);
    p += align256(BH * nblk * K * 4);
    a.cent8 = reinterpret_cast<int8_t*>(p);
    p += align256(BH * 64 * kD);
    a.cnorm = reinterpret_cast<int32_t*>(p);
  }
  return hip_status(vc::launch_group(a, (int)BH, static_cast<hipStream_t>(stream)));
}

static vc_status prep_impl(const vc_shape* shape, const vc_opts* opts, const uint16_t* Q, const uint16_t* K,
                           const uint16_t* V, const int32_t* perm, const int32_t* q_perm, const float* rope_cos,
                           const float* rope_sin, const vc_prepped* out, void* ws, size_t ws_bytes, bool use_scratch,
                           void* stream) {
  vc_status st = check_shape(shape);
  if (st != VC_OK) return st;
  if ((st = check_opts(opts)) != VC_OK) return st;
  if (!Q || !K || !V || !out) return VC_ERR_NULL;
  if (use_scratch) {
    // the workspace is this GPU's static scratch: refuse shapes that need more
    ws_bytes = kScratchBytes;
    if (prep_ws(shape) > ws_bytes) return VC_ERR_WORKSPACE;
  }
  const bool mx = opts->qk_fmt == VC_QK_MXFP4;
  // the per-block fp32 scales (INT8) or the E8M0 scale bytes (MXFP4)
  const void* qsc = mx ? (const void*)out->q_mx_scale : (const void*)out->q_scale;
  const void* ksc = mx ? (const void*)out->k_mx_scale : (const void*)out->k_scale;
  if (!out->q || !qsc || !out->k || !ksc || !out->k_mean || !out->v || !out->v_scale || !out->v_mean)
    return VC_ERR_NULL;
  if (opts->rope && (!rope_cos || !rope_sin)) return VC_ERR_NULL;
  if (!use_scratch && (!ws || ws_bytes < prep_ws(shape))) return VC_ERR_WORKSPACE;
  const void* ptrs[] = {Q, K, V, out->q, qsc, out->k, ksc, out->k_mean, out->v, out->v_scale, out->v_mean};
  for (const void* p : ptrs)
    if (!aligned16(p)) return VC_ERR_ALIGN;
  if ((perm && !aligned16(perm)) || (q_perm && !aligned16(q_perm)) || (rope_cos && !aligned16(rope_cos)) ||
      (rope_sin && !aligned16(rope_sin)) || (!use_scratch && !aligned16(ws)))
    return VC_ERR_ALIGN;
  // the last step before launching: the validation above fails the same way with and without a GPU
  if (use_scratch && (st = scratch_ptr(&ws)) != VC_OK) return st;

  vc::PrepArgs a{};
  const size_t BH = (size_t)shape->B * shape->H, T = blocks_of(shape->N, 128);
  a.Q = Q;
  a.K = K;
  a.V = V;
  a.perm = perm;
  a.q_perm = q_perm;
  a.rope_cos = rope_cos;
  a.rope_sin = rope_sin;
  a.q = out->q;
  a.q_scale = out->q_scale;
  a.k = out->k;
  a.k_scale = out->k_scale;
  a.k_mean = out->k_mean;
  a.v = out->v;
  a.v_scale = out->v_scale;
  a.v_mean = out->v_mean;
  char* p = static_cast<char*>(ws);
  a.ws_ksum = reinterpret_cast<float*>(p);
  p += align256(BH * T * kD * 4);
  a.ws_vamax = reinterpret_cast<float*>(p);
  p += align256(BH * T * kD * 4);
  a.ws_vinv = reinterpret_cast<float*>(p);
  a.N = shape->N;
  a.T = (int)T;
  a.F = shape->F;
  a.Ht = shape->Ht;
  a.Wd = shape->Wd;
  a.inv_w = 1.0f / (float)shape->Wd;
  a.inv_hw = 1.0f / (float)(shape->Ht * shape->Wd);
  a.rope = opts->rope;
  a.hadamard = opts->hadamard;
  a.smooth_k = opts->smooth_k;
  a.smooth_v = opts->smooth_v;
  a.qk_fmt = opts->qk_fmt;
  a.q_mxs = out->q_mx_scale;
  a.k_mxs = out->k_mx_scale;
  return hip_status(vc::launch_prep(a, (int)BH, static_cast<hipStream_t>(stream)));
}

vc_status vc_attn_prep(const vc_shape* shape, const vc_opts* opts, const uint16_t* Q, const uint16_t* K,
                       const uint16_t* V, const int32_t* perm, const int32_t* q_perm, const float* rope_cos,
                       const float* rope_sin, const vc_prepped* out, void* ws, size_t ws_bytes, void* stream) {
  return prep_impl(shape, opts, Q, K, V, perm, q_perm, rope_cos, rope_sin, out, ws, ws_bytes, false, stream);
}

vc_status vc_attn_prep_noalloc(const vc_shape* shape, const vc_opts* opts, const uint16_t* Q, const uint16_t* K,
                               const uint16_t* V, const int32_t* perm, const int32_t* q_perm, const float* rope_cos,
                               const float* rope_sin, const vc_prepped* out, void* stream) {
  return prep_impl(shape, opts, Q, K, V, perm, q_perm, rope_cos, rope_sin, out, nullptr, 0, true, stream);
}

static vc_status attn_forward(const vc_shape* shape, const vc_opts* opts, const vc_prepped* in, const int32_t* q_perm,
                              uint16_t* O, uint8_t* p_codes, void* stream) {
  vc_status st = check_shape(shape);
  if (st != VC_OK) return st;
  if ((st = check_opts(opts)) != VC_OK) return st;
  if (!in || !O) return VC_ERR_NULL;
  const bool mx = opts->qk_fmt == VC_QK_MXFP4;
  const void* qsc = mx ? (const void*)in->q_mx_scale : (const void*)in->q_scale;
  const void* ksc = mx ? (const void*)in->k_mx_scale : (const void*)in->k_scale;
  if (!in->q || !qsc || !in->k || !ksc || !in->v || !in->v_scale || !in->v_mean) return VC_ERR_NULL;
  const void* ptrs[] = {in->q, qsc, in->k, ksc, in->v, in->v_scale, in->v_mean, O};
  for (const void* p : ptrs)
    if (!aligned16(p)) return VC_ERR_ALIGN;
  if (q_perm && !aligned16(q_perm)) return VC_ERR_ALIGN;
  if (p_codes && !aligned16(p_codes)) return VC_ERR_ALIGN;

  vc::FwdArgs a{};
  const size_t BH = (size_t)shape->B * shape->H;
  a.q = in->q;
  a.q_scale = in->q_scale;
  a.k = in->k;
  a.k_scale = in->k_scale;
  a.v = in->v;
  a.v_scale = in->v_scale;
  a.v_mean = in->v_mean;
  a.q_perm = q_perm;
  a.O = O;
  a.p_codes = p_codes;
  a.N = shape->N;
  a.T = blocks_of(shape->N, 128);
  // score scale in log2 units: sm_scale * log2(e), with the unnormalised Hadamard's 1/128
  const double sm = opts->sm_scale > 0.f ? (double)opts->sm_scale : (double)(float)(1.0 / std::sqrt(128.0));
  double kappa = sm * 1.4426950408889634074;
  if (opts->hadamard) kappa /= 128.0;
  a.kappa = (float)kappa;
  a.cbias = 120.0f + opts->beta;
  a.p_mode = opts->p_mode;
  a.smooth_v = opts->smooth_v;
  a.qk_fmt = opts->qk_fmt;
  a.q_mxs = in->q_mx_scale;
  a.k_mxs = in->k_mx_scale;
  return hip_status(vc::launch_forward(a, (int)BH, static_cast<hipStream_t>(stream)));
}

vc_status vc_attn_forward(const vc_shape* shape, const vc_opts* opts, const vc_prepped* in, const int32_t* q_perm,
                          uint16_t* O, void* stream) {
  return attn_forward(shape, opts, in, q_perm, O, nullptr, stream);
}

vc_status vc_attn_forward_codes(const vc_shape* shape, const vc_opts* opts, const vc_prepped* in,
                                const int32_t* q_perm, uint16_t* O, uint8_t* p_codes, size_t p_codes_bytes,
                                void* stream) {
  const vc_status st = check_shape(shape);
  if (st != VC_OK) return st;
  if (!p_codes) return VC_ERR_NULL;
  const size_t need = (size_t)shape->B * shape->H * shape->N * ((size_t)blocks_of(shape->N, 128) * 128);
  if (p_codes_bytes < need) return VC_ERR_WORKSPACE;
  return attn_forward(shape, opts, in, q_perm, O, p_codes, stream);
}

vc_status vc_fp8_score_product(const uint8_t* a, const uint8_t* b, const float* c_in, float* out, int32_t n,
                               void* stream) {
  if (!a || !b || !c_in || !out) return VC_ERR_NULL;
  if (n < 1) return VC_ERR_SHAPE;
  if (!aligned16(a) || !aligned16(b) || !aligned16(c_in) || !aligned16(out)) return VC_ERR_ALIGN;
  return hip_status(vc::launch_fp8_score_product(a, b, c_in, out, n, static_cast<hipStream_t>(stream)));
}

const char* vc_status_str(vc_status s) {
  switch (s) {
    case VC_OK: return "ok";
    case VC_ERR_NULL: return "a required pointer is NULL";
    case VC_ERR_SHAPE: return "unsupported shape (d must be 128, N = F*Ht*Wd, sizes positive and bounded)";
    case VC_ERR_UNSUPPORTED: return "unsupported option value";
    case VC_ERR_WORKSPACE: return "workspace missing or too small";
    case VC_ERR_ALIGN: return "tensor pointer not 16-byte aligned";
    case VC_ERR_HIP: return "HIP launch or runtime error";
    case VC_ERR_INTERNAL: return "internal error";
  }
  return "unknown status";
}

int vc_last_hip_error(void) { return g_last_hip; }

}  // extern "C"
