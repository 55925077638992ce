// tg_gmm_update: per-pixel adaptive Gaussian-mixture background model.
//
// The RoIs the paper partitions and stitches come from a Gaussian-mixture background
// model (Sec. III-A, step 1; Sec. V). Each pixel keeps up to K isotropic RGB components
// (weight, mean, variance), heaviest first; every frame a sample is tested against them,
// owned by the heaviest close one, and the mixture adapts (Zivkovic's online form of the
// Stauffer-Grimson mixture). The per-pixel steps and their rounding are those declared
// at tg_gmm_update.
//
// The kernel is a stream over HBM: per pixel it reads the sample (3 bytes), the count of
// components in use and those components (20 bytes each), and writes them back with the
// mask. Component 0's planes are read together with the sample and the counts. State is planar (one plane per component field) so that a wave's 64 threads, four
// pixels each, load and store 1 KB contiguous runs per plane, and planes past the
// components a thread's pixels use are neither read nor written. All arithmetic uses
// explicitly rounded operations, so the foreground decisions match any binary32
// implementation of the same steps bit for bit.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "tg.h"

// Built with -ffp-contract=off: every binary32 operation here is rounded on its own (no
// multiply-add fusion), so decisions taken in floating point match any plain IEEE
// implementation of the same steps.

namespace {

constexpr int kThreads = 256;
constexpr int kPix = 4;  // pixels per thread
constexpr int kFields = 5;

typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GmmConst {
  float alpha, decay, tb, tg, var_init, var_min, var_max, ratio;
};

template <int K>
struct Mix {
  float w[K], r[K], g[K], b[K], v[K];
  int n;
};

template <int K>
__device__ __forceinline__ void swap_at(Mix<K> &c, int j) {
  float t;
  t = c.w[j]; c.w[j] = c.w[j + 1]; c.w[j + 1] = t;
  t = c.r[j]; c.r[j] = c.r[j + 1]; c.r[j + 1] = t;
  t = c.g[j]; c.g[j] = c.g[j + 1]; c.g[j + 1] = t;
  t = c.b[j]; c.b[j] = c.b[j + 1]; c.b[j + 1] = t;
  t = c.v[j]; c.v[j] = c.v[j + 1]; c.v[j + 1] = t;
}

// One sample (x0, x1, x2) into one pixel's mixture; returns the foreground flag.
template <int K>
__device__ __forceinline__ uint32_t update_pixel(Mix<K> &c, float x0, float x1, float x2,
                                                 const GmmConst &P) {
  int M = c.n;
  float d2[K];
  int owner = -1;
  bool background = false;
  float before = 0.0f;
#pragma unroll
  for (int m = 0; m < K; ++m) {
    if (m < M) {
      const float dr = __fsub_rn(x0, c.r[m]), dg = __fsub_rn(x1, c.g[m]),
                  db = __fsub_rn(x2, c.b[m]);
      float d = __fmul_rn(dr, dr);
      d = __fadd_rn(d, __fmul_rn(dg, dg));
      d = __fadd_rn(d, __fmul_rn(db, db));
      d2[m] = d;
      if (owner < 0 && d < __fmul_rn(P.tg, c.v[m])) owner = m;
      if (before <= P.ratio && d < __fmul_rn(P.tb, c.v[m])) background = true;
      before = __fadd_rn(before, c.w[m]);
    } else {
      d2[m] = 0.0f;
    }
  }

#pragma unroll
  for (int m = 0; m < K; ++m) {
    if (m < M) {
      const float o = m == owner ? 1.0f : 0.0f;
      c.w[m] = __fsub_rn(__fadd_rn(c.w[m], __fmul_rn(P.alpha, __fsub_rn(o, c.w[m]))), P.decay);
    }
    if (m == owner) {
      const float rho = __fdiv_rn(P.alpha, c.w[m]);
      c.r[m] = __fadd_rn(c.r[m], __fmul_rn(rho, __fsub_rn(x0, c.r[m])));
      c.g[m] = __fadd_rn(c.g[m], __fmul_rn(rho, __fsub_rn(x1, c.g[m])));
      c.b[m] = __fadd_rn(c.b[m], __fmul_rn(rho, __fsub_rn(x2, c.b[m])));
      float v = __fadd_rn(c.v[m], __fmul_rn(rho, __fsub_rn(d2[m], c.v[m])));
      v = v < P.var_min ? P.var_min : v;
      v = v > P.var_max ? P.var_max : v;
      c.v[m] = v;
    }
  }

  // Remove negative weights, keeping the order of the rest: a stable partition by
  // adjacent swaps, run only when some weight is negative.
  bool any_negative = false;
#pragma unroll
  for (int m = 0; m < K; ++m) any_negative |= m < M && c.w[m] < 0.0f;
  if (any_negative) {
#pragma unroll
    for (int pass = 0; pass < K - 1; ++pass) {
#pragma unroll
      for (int j = 0; j + 1 < K - pass; ++j)
        if (j + 1 < M && c.w[j] < 0.0f && !(c.w[j + 1] < 0.0f)) swap_at(c, j);
    }
    int kept = 0;
#pragma unroll
    for (int m = 0; m < K; ++m) kept += m < M && !(c.w[m] < 0.0f);
    M = kept;
  }

  if (owner < 0) {
    const int at = M < K ? M : K - 1;
#pragma unroll
    for (int m = 0; m < K; ++m)
      if (m == at) {
        c.w[m] = P.alpha;
        c.r[m] = x0;
        c.g[m] = x1;
        c.b[m] = x2;
        c.v[m] = P.var_init;
      }
    M = at + 1;
  }

  float sum = 0.0f;
#pragma unroll
  for (int m = 0; m < K; ++m)
    if (m < M) sum = __fadd_rn(sum, c.w[m]);
#pragma unroll
  for (int m = 0; m < K; ++m)
    if (m < M) c.w[m] = __fdiv_rn(c.w[m], sum);

  // Stable sort, heaviest first (bubble passes), skipped when already in order.
  bool unsorted = false;
#pragma unroll
  for (int j = 0; j + 1 < K; ++j) unsorted |= j + 1 < M && c.w[j + 1] > c.w[j];
  if (unsorted) {
#pragma unroll
    for (int pass = 0; pass < K - 1; ++pass) {
#pragma unroll
      for (int j = 0; j + 1 < K - pass; ++j)
        if (j + 1 < M && c.w[j + 1] > c.w[j]) swap_at(c, j);
    }
  }
  c.n = M;
  return background ? 0u : 1u;
}

template <int K>
__global__ __launch_bounds__(kThreads) void gmm_kernel(const uint8_t *__restrict__ frames,
                                                       float *__restrict__ state,
                                                       uint8_t *__restrict__ modes,
                                                       uint8_t *__restrict__ mask,
                                                       int64_t n_px, int64_t stride,
                                                       const GmmConst P) {
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t p0 = g * kPix;
  if (p0 >= n_px) return;

  if (p0 + kPix <= n_px) {
    // Four whole pixels: 12 sample bytes, one modes word, one float4 per used plane.
    const uint32_t *fw = reinterpret_cast<const uint32_t *>(frames + 3 * p0);
    const uint32_t s0 = __builtin_nontemporal_load(fw), s1 = __builtin_nontemporal_load(fw + 1),
                   s2 = __builtin_nontemporal_load(fw + 2);
    const uint32_t mw = *reinterpret_cast<const uint32_t *>(modes + p0);
    int n[kPix], nmax = 0;
#pragma unroll
    for (int i = 0; i < kPix; ++i) {
      n[i] = min(static_cast<int>((mw >> (8 * i)) & 0xFFu), K);
      nmax = max(nmax, n[i]);
    }
    Mix<K> c[kPix];
#pragma unroll
    for (int m = 0; m < K; ++m) {
      f32x4 f[kFields];
      // Component 0 is loaded without waiting for the counts (every pixel past its first
      // frame uses it; for a fresh pixel the values are ignored), so its loads travel
      // with the sample's and the counts' instead of one round trip later.
      if (m == 0 || m < nmax) {
#pragma unroll
        for (int q = 0; q < kFields; ++q)
          f[q] = __builtin_nontemporal_load(
              reinterpret_cast<const f32x4 *>(state + (kFields * m + q) * stride + p0));
      } else {
#pragma unroll
        for (int q = 0; q < kFields; ++q) f[q] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      }
#pragma unroll
      for (int i = 0; i < kPix; ++i) {
        c[i].w[m] = f[0][i];
        c[i].r[m] = f[1][i];
        c[i].g[m] = f[2][i];
        c[i].b[m] = f[3][i];
        c[i].v[m] = f[4][i];
      }
    }
    const uint32_t sb[3] = {s0, s1, s2};
    uint32_t out_mask = 0, out_modes = 0;
    int nmax_out = 0;
#pragma unroll
    for (int i = 0; i < kPix; ++i) {
      const int o = 3 * i;
      const float x0 = static_cast<float>((sb[o / 4] >> (8 * (o % 4))) & 0xFFu);
      const float x1 = static_cast<float>((sb[(o + 1) / 4] >> (8 * ((o + 1) % 4))) & 0xFFu);
      const float x2 = static_cast<float>((sb[(o + 2) / 4] >> (8 * ((o + 2) % 4))) & 0xFFu);
      c[i].n = n[i];
      out_mask |= update_pixel<K>(c[i], x0, x1, x2, P) << (8 * i);
      out_modes |= static_cast<uint32_t>(c[i].n) << (8 * i);
      nmax_out = max(nmax_out, c[i].n);
    }
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if (m < nmax_out) {
        f32x4 f[kFields];
#pragma unroll
        for (int i = 0; i < kPix; ++i) {
          f[0][i] = c[i].w[m];
          f[1][i] = c[i].r[m];
          f[2][i] = c[i].g[m];
          f[3][i] = c[i].b[m];
          f[4][i] = c[i].v[m];
        }
#pragma unroll
        for (int q = 0; q < kFields; ++q)
          __builtin_nontemporal_store(
              f[q], reinterpret_cast<f32x4 *>(state + (kFields * m + q) * stride + p0));
      }
    }
    *reinterpret_cast<uint32_t *>(modes + p0) = out_modes;
    *reinterpret_cast<uint32_t *>(mask + p0) = out_mask;
    return;
  }

  // The last, partial group: one pixel at a time.
  for (int64_t p = p0; p < n_px; ++p) {
    Mix<K> c;
    c.n = min(static_cast<int>(modes[p]), K);
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if (m < c.n) {
        c.w[m] = state[(kFields * m + 0) * stride + p];
        c.r[m] = state[(kFields * m + 1) * stride + p];
        c.g[m] = state[(kFields * m + 2) * stride + p];
        c.b[m] = state[(kFields * m + 3) * stride + p];
        c.v[m] = state[(kFields * m + 4) * stride + p];
      } else {
        c.w[m] = c.r[m] = c.g[m] = c.b[m] = c.v[m] = 0.0f;
      }
    }
    const uint32_t fg = update_pixel<K>(c, static_cast<float>(frames[3 * p]),
                                        static_cast<float>(frames[3 * p + 1]),
                                        static_cast<float>(frames[3 * p + 2]), P);
#pragma unroll
    for (int m = 0; m < K; ++m) {
      if (m < c.n) {
        state[(kFields * m + 0) * stride + p] = c.w[m];
        state[(kFields * m + 1) * stride + p] = c.r[m];
        state[(kFields * m + 2) * stride + p] = c.g[m];
        state[(kFields * m + 3) * stride + p] = c.b[m];
        state[(kFields * m + 4) * stride + p] = c.v[m];
      }
    }
    modes[p] = static_cast<uint8_t>(c.n);
    mask[p] = static_cast<uint8_t>(fg);
  }
}

bool params_ok(const tg_gmm_params &p) {
  return p.n_mix >= 1 && p.n_mix <= TG_GMM_MAX_MIX && p.alpha > 0.0f && p.alpha <= 1.0f &&
         p.var_min > 0.0f && p.var_min <= p.var_max && p.var_init >= p.var_min &&
         p.var_init <= p.var_max && p.complexity_reduction >= 0.0f &&
         p.complexity_reduction < 1.0f && p.var_threshold >= 0.0f &&
         p.var_threshold_gen >= 0.0f && p.background_ratio == p.background_ratio;
}

template <int K>
void launch(const tg_gmm_args *a, int64_t n_px, const GmmConst &P, hipStream_t s) {
  const int64_t groups = (n_px + kPix - 1) / kPix;
  const uint32_t blocks = static_cast<uint32_t>((groups + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(gmm_kernel<K>, dim3(blocks), dim3(kThreads), 0, s, a->frames, a->state,
                     a->modes, a->mask, n_px, tg_gmm_plane_stride(n_px), P);
}

}  // namespace

extern "C" int64_t tg_gmm_plane_stride(int64_t n_px) {
  return n_px <= 0 ? 0 : (n_px + 63) / 64 * 64;
}

extern "C" size_t tg_gmm_state_bytes(int64_t n_px, int32_t n_mix) {
  if (n_px <= 0 || n_mix < 1 || n_mix > TG_GMM_MAX_MIX) return 0;
  return sizeof(float) * kFields * static_cast<size_t>(n_mix) *
         static_cast<size_t>(tg_gmm_plane_stride(n_px));
}

extern "C" int tg_gmm_update(const tg_gmm_args *a, void *stream) {
  if (!a || a->n_frames < 0 || a->width < 1 || a->height < 1 || !params_ok(a->params))
    return TG_E_INVAL;
  if (a->n_frames == 0) return TG_OK;
  if (!a->frames || !a->state || !a->modes || !a->mask) return TG_E_INVAL;
  if (reinterpret_cast<uintptr_t>(a->frames) % 4 || reinterpret_cast<uintptr_t>(a->state) % 16 ||
      reinterpret_cast<uintptr_t>(a->modes) % 4 || reinterpret_cast<uintptr_t>(a->mask) % 4)
    return TG_E_INVAL;
  const int64_t n_px = int64_t(a->n_frames) * a->width * a->height;
  if ((n_px + kPix - 1) / kPix > int64_t(kThreads) * 0x7FFFFFFF) return TG_E_INVAL;
  const tg_gmm_params &p = a->params;
  GmmConst P;
  P.alpha = p.alpha;
  P.decay = p.alpha * p.complexity_reduction;  // alpha c_T: one binary32 product
  P.tb = p.var_threshold;
  P.tg = p.var_threshold_gen;
  P.var_init = p.var_init;
  P.var_min = p.var_min;
  P.var_max = p.var_max;
  P.ratio = p.background_ratio;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (p.n_mix) {
    case 1: launch<1>(a, n_px, P, s); break;
    case 2: launch<2>(a, n_px, P, s); break;
    case 3: launch<3>(a, n_px, P, s); break;
    case 4: launch<4>(a, n_px, P, s); break;
    default: launch<5>(a, n_px, P, s); break;
  }
  return hipGetLastError() == hipSuccess ? TG_OK : TG_E_HIP;
}
