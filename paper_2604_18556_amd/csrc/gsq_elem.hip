// Elementwise kernels of the GSQ layer step on gfx950: initialisation (Eq. 4, App. A),
// the Gumbel-Softmax sample of Alg. 1 and its residual, the fused gradient + Adam pass,
// hardening (argmax of Alg. 2) and bit-packing.
//
// Data layout in HBM: logits and both optimiser moments are K planes of fp32 values, laid out
// in blocks of kStateBlock coordinates (row-major over B*O*I) with the K planes of a block side
// by side, so every plane streams with 16-byte loads across a wavefront and a wavefront's planes
// lie close together in memory.  A wavefront owns 256 consecutive columns of one row; lane l
// owns columns 4l..4l+3.  Scale groups (16..256 columns) therefore lie inside one wavefront and
// their gradient is reduced with lane shuffles in a fixed order.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <type_traits>

#include "gsq_device.hpp"
#include "gsq_internal.h"

namespace gsq {
namespace {

constexpr int kBlock = 256;   // 4 wavefronts
constexpr int kCols = 256;    // columns per wavefront

template <bool kF64>
using Real = typename std::conditional<kF64, double, float>::type;

__device__ __forceinline__ float f4get(const float4& v, int q) {
  return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
}

__device__ __forceinline__ void f4set(float4& v, int q, float x) {
  if (q == 0) v.x = x; else if (q == 1) v.y = x; else if (q == 2) v.z = x; else v.w = x;
}

__device__ __forceinline__ bool finite4(const float4& v) {
  return __builtin_isfinite(v.x) && __builtin_isfinite(v.y) && __builtin_isfinite(v.z) &&
         __builtin_isfinite(v.w);
}

// Float offset of logit (or moment) k of coordinate e in the blocked state layout.  Four
// consecutive coordinates from a multiple of 4 lie in one block, so a lane's float4 is
// contiguous and 16-byte aligned.
__device__ __forceinline__ int64_t state_off(int64_t e, int k, int K) {
  return (e / kStateBlock) * (K * kStateBlock) + (int64_t)k * kStateBlock + (e % kStateBlock);
}

// Streaming accesses of the state and G: each is touched once per launch, so the loads and
// stores carry the non-temporal hint (no cache allocation).  On the backward's access pattern
// this moves 14-21 % more bytes per second than plain accesses.  W and R keep plain accesses:
// R is read next by the contraction, and the hint on them measured slightly slower.
__device__ __forceinline__ float4 ld_stream(const float* p) {
  float4 v;
  v.x = __builtin_nontemporal_load(p);
  v.y = __builtin_nontemporal_load(p + 1);
  v.z = __builtin_nontemporal_load(p + 2);
  v.w = __builtin_nontemporal_load(p + 3);
  return v;
}

__device__ __forceinline__ void st_stream(float* p, const float4& v) {
  __builtin_nontemporal_store(v.x, p);
  __builtin_nontemporal_store(v.y, p + 1);
  __builtin_nontemporal_store(v.z, p + 2);
  __builtin_nontemporal_store(v.w, p + 3);
}

__device__ __forceinline__ void load_w4(const void* W, int w_bf16, int64_t e, float (&w)[4]) {
  if (w_bf16) {
    const uint2 u = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(W) + e);
    w[0] = __uint_as_float(u.x << 16);
    w[1] = __uint_as_float(u.x & 0xFFFF0000u);
    w[2] = __uint_as_float(u.y << 16);
    w[3] = __uint_as_float(u.y & 0xFFFF0000u);
  } else {
    const float4 v = *reinterpret_cast<const float4*>(static_cast<const float*>(W) + e);
    w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
  }
}

// R is stored in the contraction's padded layout: row (b, o) at (b*Opad + o)*Ipad.
__device__ __forceinline__ int64_t padded_index(const ElemArgs& a, int64_t row, int64_t col) {
  const int64_t b = row / a.O;
  return (b * a.Opad + (row - b * a.O)) * a.Ipad + col;
}

template <bool kF64>
__device__ __forceinline__ void store_r4(void* R, int64_t idx, const float (&r)[4]) {
  if constexpr (kF64) {
    *reinterpret_cast<float4*>(static_cast<float*>(R) + idx) = make_float4(r[0], r[1], r[2], r[3]);
  } else {
    uint2 u;
    u.x = (uint32_t)bf16_rne(r[0]) | ((uint32_t)bf16_rne(r[1]) << 16);
    u.y = (uint32_t)bf16_rne(r[2]) | ((uint32_t)bf16_rne(r[3]) << 16);
    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(R) + idx) = u;
  }
}

// R = W - s v before the contraction's rounding; the forward, the fused next sample and the
// backward's loss all form it with this one expression.
template <bool kF64>
__device__ __forceinline__ float residual(float w, Real<kF64> s, Real<kF64> v) {
  return (float)((Real<kF64>)w - s * v);
}

// fp32 path: hardware exp2 / reciprocal / square root (about 1 ulp); fp64 path: libm.
constexpr float kLog2e = 1.4426950408889634f;
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float fast_sqrt(float x) { return __builtin_amdgcn_sqrtf(x); }

// One coordinate's relaxed sample (Alg. 1): p = softmax((kappa l + g) / tau), with the
// largest perturbed logit r subtracted first.  vp = sum_k p_k (c_k - c_r), so that the soft
// level v = c_r + vp and c_k - v = (c_k - c_r) - vp keep full relative accuracy when one
// level holds almost all the mass.  c holds the values the K logits stand for.
template <int K, bool kF64>
__device__ __forceinline__ void soft_sample(const float (&l)[K], const float (&c)[K], const float (&g)[K],
                                            float kappa, Real<kF64> inv_tau, Real<kF64> (&p)[K],
                                            Real<kF64>& vp, Real<kF64>& cr) {
  using T = Real<kF64>;
  T b[K];
#pragma unroll
  for (int k = 0; k < K; ++k) b[k] = (T)kappa * (T)l[k] + (T)g[k];
  T bmax = b[0];
  cr = (T)c[0];
#pragma unroll
  for (int k = 1; k < K; ++k) {
    if (b[k] > bmax) { bmax = b[k]; cr = (T)c[k]; }
  }
  T z = 0;
  if constexpr (kF64) {
#pragma unroll
    for (int k = 0; k < K; ++k) { p[k] = exp((b[k] - bmax) * inv_tau); z += p[k]; }
  } else {
    const float s2 = inv_tau * kLog2e;   // exp(a) = exp2(a log2 e)
#pragma unroll
    for (int k = 0; k < K; ++k) { p[k] = __builtin_amdgcn_exp2f((b[k] - bmax) * s2); z += p[k]; }
  }
  T rz;
  if constexpr (kF64) rz = T(1) / z; else rz = fast_rcp(z);
  vp = 0;
#pragma unroll
  for (int k = 0; k < K; ++k) { p[k] *= rz; vp += p[k] * ((T)c[k] - cr); }
}

// Two-value relaxation with logits {-l, l} (§3): p1 = softmax over (-kappa l + g0,
// kappa l + g1) / tau, i.e. a sigmoid of (2 kappa l + g1 - g0) / tau.  The pair's noise dn is
// drawn as the difference g1 - g0 itself (a logistic value).  The smaller probability is formed
// as e / (1 + e) with e = exp(-|a|), never as 1 - p.
template <bool kF64>
__device__ __forceinline__ void pair_probs(float l, float dn, float kappa, Real<kF64> inv_tau,
                                           Real<kF64>& p0, Real<kF64>& p1) {
  using T = Real<kF64>;
  const T d = (T)2 * (T)kappa * (T)l + (T)dn;
  const T a = d * inv_tau;
  T e, big;
  if constexpr (kF64) {
    e = exp(-fabs(a));
    big = T(1) / (T(1) + e);
  } else {
    e = __builtin_amdgcn_exp2f(-fabsf(a) * kLog2e);
    big = fast_rcp(1.f + e);
  }
  const T small = e * big;
  p1 = a >= T(0) ? big : small;
  p0 = a >= T(0) ? small : big;
}

// Noise values per coordinate and draw: one Gumbel value per logit of a categorical, or one
// logistic value per binary pair (the mask's, then the sign's).
template <int K, int kMode>
constexpr int noise_count() { return kMode == GSQ_RELAX_TERNARY ? 2 : K; }

template <int kMode>
constexpr int noise_kind() { return kMode == GSQ_RELAX_TERNARY ? kLogistic : kGumbel; }

// One coordinate's relaxed sample in any relaxation: the soft level v (W_hat = s v) and
// jac[k] = (tau / kappa) dv/dl_k.
//   GRID / SHIFT: v = sum_k p_k c_k, jac[k] = p_k (c_k - v).
//   TERNARY: v = m~ b~ with m~ = p1 of the mask pair (values 0, 1) and b~ = p1 - p0 of the
//   sign pair (values -1, 1); a pair with logits {-l, l} and values (y0, y1) has
//   (tau / kappa) dy/dl = 2 p0 p1 (y1 - y0), so jac = (2 p0 p1 b~, 4 p0 p1 m~).
template <int K, int Z, bool kF64, int kMode>
__device__ __forceinline__ void coord_sample(const float (&l)[K], const float (&c)[K], const float (&g)[Z],
                                             float kappa, Real<kF64> inv_tau, Real<kF64>& v,
                                             Real<kF64> (&jac)[K]) {
  using T = Real<kF64>;
  if constexpr (kMode == GSQ_RELAX_TERNARY) {
    static_assert(K == 2 && Z == 2, "ternary: two logits, one noise value per pair");
    T pm0, pm1, pb0, pb1;
    pair_probs<kF64>(l[0], g[0], kappa, inv_tau, pm0, pm1);
    pair_probs<kF64>(l[1], g[1], kappa, inv_tau, pb0, pb1);
    const T m = pm1, b = pb1 - pb0;
    v = m * b;
    jac[0] = b * (T(2) * pm0 * pm1);
    jac[1] = m * (T(4) * pb0 * pb1);
  } else {
    static_assert(K == Z, "one noise value per logit");
    T p[K], vp, cr;
    soft_sample<K, kF64>(l, c, g, kappa, inv_tau, p, vp, cr);
    v = cr + vp;
#pragma unroll
    for (int k = 0; k < K; ++k) jac[k] = p[k] * (((T)c[k] - cr) - vp);
  }
}

// Local-shift windows in LDS: row j (a grid index) holds the levels of the five shifts around
// it, c[clip(j + k - 2, 0, n - 1)] for k < 5, padded to 8 floats.  Rows past the grid are
// filled like the last one, so a clamped index never reads an unset row.
constexpr int kWinRow = 8;
__device__ __forceinline__ void fill_windows(float* win, const ElemArgs& a) {
  for (int i = threadIdx.x; i < GSQ_MAX_LEVELS * kWinRow; i += blockDim.x) {
    const int j = i / kWinRow, k = i % kWinRow;
    int idx = j + k - 2;
    idx = idx < 0 ? 0 : idx;
    idx = idx > a.n_grid - 1 ? a.n_grid - 1 : idx;
    float v = 0.f;
#pragma unroll
    for (int m = 0; m < GSQ_MAX_LEVELS; ++m) v = (m == idx) ? a.c[m] : v;
    win[i] = k < GSQ_SHIFT_WINDOW ? v : 0.f;
  }
  __syncthreads();
}

// Base indices of the chunk's four coordinates (local shift; one byte each), or 0.
template <int kMode>
__device__ __forceinline__ uint32_t chunk_bases(const ElemArgs& a, int64_t e0) {
  if constexpr (kMode == GSQ_RELAX_SHIFT) return *reinterpret_cast<const uint32_t*>(a.J0 + e0);
  else return 0u;
}

// The values the logits of coordinate q of the chunk stand for: the grid (GRID), or the
// window of its base index read from the LDS table (SHIFT; read where needed rather than
// held in registers).
template <int K, int kMode>
__device__ __forceinline__ void coord_candidates(float (&cand)[K], const ElemArgs& a, const float* win,
                                                 uint32_t j4, int q) {
  if constexpr (kMode == GSQ_RELAX_SHIFT) {
    static_assert(K == GSQ_SHIFT_WINDOW, "five shifts");
    int j = (int)((j4 >> (8 * q)) & 0xFFu);
    j = j < a.n_grid ? j : a.n_grid - 1;          // a corrupt index cannot leave the table
    const float4 lo = *reinterpret_cast<const float4*>(win + j * kWinRow);
    cand[0] = lo.x; cand[1] = lo.y; cand[2] = lo.z; cand[3] = lo.w;
    cand[4] = win[j * kWinRow + 4];
  } else {
#pragma unroll
    for (int k = 0; k < K; ++k) cand[k] = a.c[k];
  }
}

// Noise of the thread's chunk of four coordinates (or zeros when sampling is off).
template <int Z, bool kF64, int kMode>
__device__ __forceinline__ void chunk_noise(float (&g)[4][Z], const ElemArgs& a, uint64_t e0,
                                            uint32_t t, uint32_t sample) {
  if (a.noise) {
    draw_chunk<Z, kF64, noise_kind<kMode>()>(g, a.seed, e0, t, sample);
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int k = 0; k < Z; ++k) g[q][k] = 0.f;
  }
}

// ------------------------------------------------------------------ forward: R = W - s * v
template <int K, bool kF64, int kMode>
__global__ __launch_bounds__(kBlock) void k_forward(ElemArgs a) {
  using T = Real<kF64>;
  constexpr int Z = noise_count<K, kMode>();
  __shared__ __align__(16) float win[kMode == GSQ_RELAX_SHIFT ? GSQ_MAX_LEVELS * kWinRow : 4];
  if constexpr (kMode == GSQ_RELAX_SHIFT) fill_windows(win, a);
  const int lane = threadIdx.x & 63;
  const int64_t col0 = (int64_t)blockIdx.x * kCols + lane * 4;
  const T inv_tau = kF64 ? (T)a.inv_tau_d : (T)a.inv_tau;
  const int64_t gpr = a.I / a.gs;
  for (int64_t row = (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6); row < a.rows;
       row += (int64_t)gridDim.y * 4) {
    if (col0 >= a.I) continue;
    const int64_t e0 = row * a.I + col0;
    const T s = (T)a.S[row * gpr + col0 / a.gs];
    float w[4];
    load_w4(a.W, a.w_bf16, e0, w);
    float4 lv[K];
#pragma unroll
    for (int k = 0; k < K; ++k) lv[k] = *reinterpret_cast<const float4*>(a.L + state_off(e0, k, K));
    const uint32_t j4 = chunk_bases<kMode>(a, e0);
    float g[4][Z];
    chunk_noise<Z, kF64, kMode>(g, a, (uint64_t)e0, a.t, (uint32_t)a.sample);
    float r[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float l[K], cand[K];
#pragma unroll
      for (int k = 0; k < K; ++k) l[k] = f4get(lv[k], q);
      coord_candidates<K, kMode>(cand, a, win, j4, q);
      T v, jac[K];
      coord_sample<K, Z, kF64, kMode>(l, cand, g[q], a.kappa, inv_tau, v, jac);
      r[q] = residual<kF64>(w[q], s, v);
    }
    store_r4<kF64>(a.Rout, padded_index(a, row, col0), r);
  }
}

// One parameter's optimiser update.  Adam: bias-corrected (step = lr / (1 - b1^n),
// rbc2 = 1 / sqrt(1 - b2^n)), plus decoupled decay lr wd theta (AdamW).  Lion: the sign of
// b1 m + (1 - b1) d, plus decoupled decay; the moment then moves with b2; v is untouched.
template <bool kF64, bool kLion>
__device__ __forceinline__ void opt_update(Real<kF64> d, Real<kF64>& th, Real<kF64>& m,
                                           Real<kF64>& v, Real<kF64> lr, Real<kF64> step,
                                           Real<kF64> b1, Real<kF64> b2, Real<kF64> omb1,
                                           Real<kF64> omb2, Real<kF64> rbc2, Real<kF64> eps,
                                           Real<kF64> wd) {
  using T = Real<kF64>;
  if constexpr (kLion) {
    const T c = b1 * m + omb1 * d;
    const T sg = (T)((c > T(0)) - (c < T(0)));
    th = th - lr * (sg + wd * th);
    m = b2 * m + omb2 * d;
  } else {
    m = b1 * m + omb1 * d;
    v = b2 * v + omb2 * d * d;
    if constexpr (kF64) th = th - (step * m / (sqrt(v) * rbc2 + eps) + lr * wd * th);
    else th = th - (step * m * fast_rcp(fast_sqrt(v) * rbc2 + eps) + lr * wd * th);
  }
}

// x shifted up by n lanes within each 16-lane row (lanes below the row start read 0).
template <int kCtrl>
__device__ __forceinline__ double dpp_shr(double x) {
  const uint64_t b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, kCtrl, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), kCtrl, 0xF, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

// x from lane 15 of the previous 16-lane row (kCtrl = row broadcast 15) or from lane 31
// (row broadcast 31), added only in the rows of kRows; other lanes read 0.
template <int kCtrl, int kRows>
__device__ __forceinline__ double dpp_bcast(double x) {
  const uint64_t b = __double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, kCtrl, kRows, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), kCtrl, kRows, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

// Sum over the wavefront in a fixed order, left in lane 63: prefix sums within each 16-lane
// row (shifts by 1, 2, 4, 8), then row 0's total into row 1 and row 2's into row 3, then the
// first half's total into the second half.
__device__ __forceinline__ double wave_sum_to_lane63(double x) {
  x += dpp_shr<0x111>(x);
  x += dpp_shr<0x112>(x);
  x += dpp_shr<0x114>(x);
  x += dpp_shr<0x118>(x);
  x += dpp_bcast<0x142, 0xA>(x);
  x += dpp_bcast<0x143, 0xC>(x);
  return x;
}

// ------------------------------------------------------------------ gradient + update (+ next sample)
// dL/dl_k = (kappa / tau) G s p_k (c_k - v); dL/ds = sum over the group of G v.  Adam (bias
// correction at step n = t + 1) or Lion.  With a.fuse, the sample of step t + 1 is drawn from
// the updated logits and scale and its residual written to a.Rout.  With a.want_loss, the
// loss terms R * P = R * (-G / 2) of this step's sample(s) are summed per row and 256-column
// block (R rebuilt exactly as the contraction saw it) into a.loss_part.
// Register budget of the backward.  Updating the moments one logit plane at a time (each
// plane's m and v loaded just before its update) keeps 8K fewer registers live than loading
// them all first, at the price of less memory parallelism within a wavefront.  It buys another
// wavefront per SIMD (2 -> 3) for grids of 5 to 7 levels, which keep it.  The local shift keeps
// every moment in flight: with the non-temporal state accesses that is 7-8 % faster than the
// plane-by-plane update at three wavefronts (4096 x 14336: 1.33 -> 1.23 ms; the MoE experts with
// frozen scales: 21.3 -> 19.7 ms).  The 8-level grids keep every moment in flight at two
// wavefronts: 1 % faster on the super-block MoE than the plane-by-plane update under a bound of
// three wavefronts, and with trained scales that bound spills.  The smaller grids keep all
// moments in flight as well.
template <int K, int kMode>
constexpr bool backward_plane_update() {
  return kMode == GSQ_RELAX_GRID && K >= 5 && K <= 7;
}

// Moments staged in LDS: the moment planes of a row go from HBM straight into a per-wavefront
// LDS area (global_load_lds, no registers held) right after the logits, W and G are requested,
// so their latency passes during the sample arithmetic; after the sample loop each plane is
// read back from LDS.  LDS per workgroup: 4 wavefronts x (K or 2K planes) x 1 KB.  Used where
// it measured faster: Lion over an 8-level grid, whose kernel then holds 150 instead of 184
// registers and runs three wavefronts per SIMD (4096 x 14336: 1.55 -> 1.45 ms; the MoE experts:
// 23.7 -> 22.5 ms).  Under Adam the 8-level kernel stays at two wavefronts (its 64 KB of LDS
// per workgroup) and staging was 0-5 % slower, as it was for the smaller grids, the local shift
// and the ternary pairs under either optimiser (1-4 %).
template <int K, int kMode, bool kLion>
constexpr bool backward_stage_moments() {
  return kLion && kMode == GSQ_RELAX_GRID && K == 8;
}
constexpr int kAuxNT = 2;   // cache policy of a global_load_lds: non-temporal

// Wait until every vector-memory load of this wavefront has landed (the staged moments),
// leaving the LDS and scalar counters alone; the fences keep the compiler from moving memory
// accesses across the wait.
__device__ __forceinline__ void wait_all_vm_loads() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));   // vmcnt(0)
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <int K, bool kF64, bool kScales, bool kMulti, int kMode, bool kLion>
__global__ __launch_bounds__(kBlock) void k_backward(
    ElemArgs a) {
  using T = Real<kF64>;
  constexpr int Z = noise_count<K, kMode>();
  __shared__ __align__(16) float win[kMode == GSQ_RELAX_SHIFT ? GSQ_MAX_LEVELS * kWinRow : 4];
  if constexpr (kMode == GSQ_RELAX_SHIFT) fill_windows(win, a);
  constexpr bool kStage = backward_stage_moments<K, kMode, kLion>();
  constexpr int kStagePlanes = kLion ? K : 2 * K;   // m (and v) planes of one row
  __shared__ __align__(16) float4 stage[kStage ? (kBlock / 64) * kStagePlanes * 64 : 1];
  float4* const sw = stage + (kStage ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) *
                                           (kStagePlanes * 64) : 0);
  const int lane = threadIdx.x & 63;
  const int64_t col0 = (int64_t)blockIdx.x * kCols + lane * 4;
  const bool active = col0 < a.I;
  const T inv_tau = kF64 ? (T)a.inv_tau_d : (T)a.inv_tau;
  const T kt = (T)a.kappa * inv_tau;
  const T b1 = (T)a.b1, b2 = (T)a.b2, omb1 = T(1) - (T)a.b1, omb2 = T(1) - (T)a.b2;
  const T eps = (T)a.eps;
  const T step_l = kF64 ? (T)a.step_l_d : (T)a.step_l;
  const T rbc2 = kF64 ? (T)a.rbc2_d : (T)a.rbc2;
  const T lr = (T)a.lr, wd = (T)a.wd;
  constexpr bool lion = kLion;
  const int lpg = a.gs / 4;   // lanes per scale group
  const int64_t gpr = a.I / a.gs;
  bool bad = false;
  for (int64_t row = (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6); row < a.rows;
       row += (int64_t)gridDim.y * 4) {
    const int64_t e0 = row * a.I + (active ? col0 : 0);
    const int64_t sidx = row * gpr + (active ? col0 / a.gs : 0);
    const float s32 = a.S[sidx];
    const T s = (T)s32;
    float4 lv[K];
    const int64_t gidx = active ? padded_index(a, row, col0) : 0;
#pragma unroll
    for (int k = 0; k < K; ++k)
      lv[k] = active ? ld_stream(a.L + state_off(e0, k, K))
                     : make_float4(0.f, 0.f, 0.f, 0.f);
    const uint32_t j4 = chunk_bases<kMode>(a, e0);
    float w[4] = {0.f, 0.f, 0.f, 0.f};
    if (active && (a.want_loss || a.fuse)) load_w4(a.W, a.w_bf16, e0, w);
    // the first sample's G before the staged moments: loads complete in issue order, so the
    // sample loop then waits only for the loads it uses
    const float4 gv0 = active ? ld_stream(a.G + gidx) : make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (kStage) {
      if (active) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int64_t o = state_off(e0, k, K);
          __builtin_amdgcn_global_load_lds(a.M + o, sw + k * 64, 16, 0, kAuxNT);
          if constexpr (!kLion)
            __builtin_amdgcn_global_load_lds(a.V + o, sw + (K + k) * 64, 16, 0, kAuxNT);
        }
      }
    }
    T lacc = 0;   // sum of R G over the thread's coordinates and samples
    // gradient, averaged over the step's independent samples (one unless kMulti)
    T ds_part = 0;
    T dacc[4][K];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int k = 0; k < K; ++k) dacc[q][k] = 0;
    const int M = kMulti ? a.samples : 1;
    for (int smp = 0; smp < M; ++smp) {
      const float4 gv = smp == 0 ? gv0
                        : active ? ld_stream(a.G + smp * a.g_stride + gidx)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
      float g[4][Z];
      chunk_noise<Z, kF64, kMode>(g, a, (uint64_t)e0, a.t, (uint32_t)smp);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float l[K], cand[K];
#pragma unroll
        for (int k = 0; k < K; ++k) l[k] = f4get(lv[k], q);
        coord_candidates<K, kMode>(cand, a, win, j4, q);
        T v, jac[K];
        coord_sample<K, Z, kF64, kMode>(l, cand, g[q], a.kappa, inv_tau, v, jac);
        const T gq = (T)f4get(gv, q);
        ds_part += gq * v;
        const T coef = kt * (gq * s);
#pragma unroll
        for (int k = 0; k < K; ++k) dacc[q][k] += coef * jac[k];
        if (a.want_loss) {
          float r = residual<kF64>(w[q], s, v);
          if constexpr (!kF64) r = bf16_to_f32(bf16_rne(r));
          lacc += (T)r * gq;
        }
      }
    }
    if (a.want_loss) {
      // P = -G / 2; the wavefront's sum (one row, 256 columns) in a fixed order
      const double lsum = wave_sum_to_lane63(-0.5 * (double)lacc);
      if (lane == 63) a.loss_part[row * gridDim.x + blockIdx.x] = lsum;
    }
    if constexpr (kMulti) {
      const T inv_m = T(1) / (T)M;
      ds_part *= inv_m;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int k = 0; k < K; ++k) dacc[q][k] *= inv_m;
    }
    // the moments are needed only by the update: loading them here keeps them out of the
    // registers of the sample loop
    if constexpr (kStage || backward_plane_update<K, kMode>()) {
      if constexpr (kStage) wait_all_vm_loads();
#pragma unroll
      for (int k = 0; k < K; ++k) {
        float4 mk, vk = make_float4(0.f, 0.f, 0.f, 0.f);
        if constexpr (kStage) {
          mk = active ? sw[k * 64 + lane] : make_float4(0.f, 0.f, 0.f, 0.f);
          if constexpr (!kLion)
            vk = active ? sw[(K + k) * 64 + lane] : make_float4(0.f, 0.f, 0.f, 0.f);
        } else {
          mk = active ? ld_stream(a.M + state_off(e0, k, K)) : make_float4(0.f, 0.f, 0.f, 0.f);
          if (active && !lion) vk = ld_stream(a.V + state_off(e0, k, K));
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          T th = (T)f4get(lv[k], q), m1 = (T)f4get(mk, q), v1 = (T)f4get(vk, q);
          opt_update<kF64, kLion>(dacc[q][k], th, m1, v1, lr, step_l, b1, b2, omb1, omb2, rbc2,
                           eps, wd);
          f4set(mk, q, (float)m1);
          f4set(vk, q, (float)v1);
          f4set(lv[k], q, (float)th);
        }
        if (active) {
          // a non-finite gradient reaches v under Adam, and m under Lion (whose step is only
          // a sign and stays finite)
          bad |= !(finite4(lv[k]) && finite4(lion ? mk : vk));
          const int64_t o = state_off(e0, k, K);
          st_stream(a.L + o, lv[k]);
          st_stream(a.M + o, mk);
          if (!lion) st_stream(a.V + o, vk);
        }
      }
    } else {
      float4 mv[K], vv[K];
#pragma unroll
      for (int k = 0; k < K; ++k) {
        mv[k] = active ? ld_stream(a.M + state_off(e0, k, K))
                       : make_float4(0.f, 0.f, 0.f, 0.f);
        vv[k] = (active && !lion) ? ld_stream(a.V + state_off(e0, k, K))
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int k = 0; k < K; ++k) {
          T th = (T)f4get(lv[k], q), m1 = (T)f4get(mv[k], q), v1 = (T)f4get(vv[k], q);
          opt_update<kF64, kLion>(dacc[q][k], th, m1, v1, lr, step_l, b1, b2, omb1, omb2, rbc2,
                           eps, wd);
          f4set(mv[k], q, (float)m1);
          f4set(vv[k], q, (float)v1);
          f4set(lv[k], q, (float)th);
        }
      if (active) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
          bad |= !(finite4(lv[k]) && finite4(lion ? mv[k] : vv[k]));
          const int64_t o = state_off(e0, k, K);
          st_stream(a.L + o, lv[k]);
          st_stream(a.M + o, mv[k]);
          if (!lion) st_stream(a.V + o, vv[k]);
        }
      }
    }
    float s_new = s32;
    if constexpr (kScales) {
      // fixed-order butterfly over the lanes of the group; the group's first lane owns the sum
      for (int off = 1; off < lpg; off <<= 1) ds_part += __shfl_xor(ds_part, off, 64);
      const bool leader = active && (lane & (lpg - 1)) == 0;
      if (leader) {
        const T step_s = kF64 ? (T)a.step_s_d : (T)a.step_s;
        T th = s, m1 = (T)a.MS[sidx], v1 = (T)a.VS[sidx];
        opt_update<kF64, kLion>(ds_part, th, m1, v1, (T)a.lr_s, step_s, b1, b2, omb1, omb2, rbc2,
                         eps, wd);
        s_new = (float)th;
        bad |= !(__builtin_isfinite(s_new) && __builtin_isfinite((float)(lion ? m1 : v1)));
        a.MS[sidx] = (float)m1;
        a.VS[sidx] = (float)v1;
        a.S[sidx] = s_new;
      }
      s_new = __shfl(s_new, lane & ~(lpg - 1), 64);
    }
    if (a.fuse && active) {
      const T inv_tau_n = kF64 ? (T)a.inv_tau_n_d : (T)a.inv_tau_n;
      float g[4][Z];
      chunk_noise<Z, kF64, kMode>(g, a, (uint64_t)e0, a.t_next, 0u);
      float r[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float l[K], cand[K];
#pragma unroll
        for (int k = 0; k < K; ++k) l[k] = f4get(lv[k], q);
        coord_candidates<K, kMode>(cand, a, win, j4, q);
        T v, jac[K];
        coord_sample<K, Z, kF64, kMode>(l, cand, g[q], a.kappa_n, inv_tau_n, v, jac);
        r[q] = residual<kF64>(w[q], (T)s_new, v);
      }
      store_r4<kF64>(a.Rout, padded_index(a, row, col0), r);
    }
  }
  if (bad) *a.flag = 1;
}

// ------------------------------------------------------------------ initialisation
__global__ void k_symmetrize(const float* __restrict__ Hin, void* Hout, int64_t I, int64_t Ipad,
                             int bf16) {
  __shared__ float tile[32][33];
  const int64_t b = blockIdx.z;
  const int64_t i0 = (int64_t)blockIdx.y * 32, j0 = (int64_t)blockIdx.x * 32;
  const float* H = Hin + b * I * I;
  for (int r = threadIdx.y; r < 32; r += 8) {
    const int64_t j = j0 + r, i = i0 + threadIdx.x;
    tile[r][threadIdx.x] = (j < I && i < I) ? H[j * I + i] : 0.f;
  }
  __syncthreads();
  for (int r = threadIdx.y; r < 32; r += 8) {
    const int64_t i = i0 + r, j = j0 + threadIdx.x;
    const float x = (i < I && j < I) ? H[i * I + j] : 0.f;
    const float sym = (x + tile[threadIdx.x][r]) * 0.5f;
    const int64_t o = b * Ipad * Ipad + i * Ipad + j;
    if (bf16) static_cast<uint16_t*>(Hout)[o] = bf16_rne(sym);
    else static_cast<float*>(Hout)[o] = sym;
  }
}

__device__ __forceinline__ float load_w1(const void* W, int w_bf16, int64_t e) {
  return w_bf16 ? bf16_to_f32(static_cast<const uint16_t*>(W)[e]) : static_cast<const float*>(W)[e];
}

// s = max|W_group| / max|c| (IEEE division), 1 for an all-zero group.
__global__ void k_init_scales_group(const void* W, int w_bf16, float* S, int64_t ngroups, int gs,
                                    float cmax) {
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < ngroups;
       g += (int64_t)gridDim.x * blockDim.x) {
    float amax = 0.f;
    for (int i = 0; i < gs; ++i) amax = fmaxf(amax, fabsf(load_w1(W, w_bf16, g * gs + i)));
    const float s = __fdiv_rn(amax, cmax);
    S[g] = s == 0.f ? 1.f : s;
  }
}

// 256-weight super-block: d = fp16(max_j s_j / 63), sc_j = clamp(rint(s_j / d), 0, 63),
// effective scale d * sc_j per 16-weight sub-block.
__global__ void k_init_scales_superblock(const void* W, int w_bf16, float* S, uint16_t* D,
                                         uint8_t* SC, int64_t nblocks, float cmax) {
  for (int64_t sb = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; sb < nblocks;
       sb += (int64_t)gridDim.x * blockDim.x) {
    float raw[16];
    float mx = 0.f;
    for (int j = 0; j < 16; ++j) {
      float amax = 0.f;
      for (int i = 0; i < 16; ++i) amax = fmaxf(amax, fabsf(load_w1(W, w_bf16, sb * 256 + j * 16 + i)));
      raw[j] = __fdiv_rn(amax, cmax);
      mx = fmaxf(mx, raw[j]);
    }
    const __half dh = __float2half_rn(__fdiv_rn(mx, 63.f));
    const float d = __half2float(dh);
    D[sb] = __half_as_ushort(dh);
    for (int j = 0; j < 16; ++j) {
      const float q = d > 0.f ? __fdiv_rn(raw[j], d) : 0.f;
      const float scq = fminf(fmaxf(rintf(q), 0.f), 63.f);
      SC[sb * 16 + j] = (uint8_t)scq;
      S[sb * 16 + j] = d * scq;
    }
  }
}

struct InitConsts {
  float c[GSQ_MAX_LEVELS];
  double mids[GSQ_MAX_LEVELS];   // (c_k + c_{k+1}) / 2, exact in fp64
  int K;                         // logits per coordinate
  int n_grid;
  int relax;
  float alpha, sigma;
  int noise;
  uint64_t seed;
};

// Round-to-nearest code q (fp32 ratio, ties to the lower level), then the warm-start logits
// around it plus Eq. 4's N(0,1) noise (Box-Muller on Philox stream 1):
// l = sigma_init * (eps + alpha * prior).
//   GRID: prior_k = -(c_k - c_q)^2 / 2, mean-subtracted (App. A);
//   SHIFT: j0 = q and prior_k = -delta_k^2 / 2, mean-subtracted (App. A, b > 2);
//   TERNARY: Eq. 3, prior = (q != 0 ? 1 : -1, sign of q) for the level c_q in {-1, 0, 1}.
// fp64 arithmetic, fp32 storage.
__global__ void k_init_logits(const void* W, int w_bf16, const float* S, float* L, uint8_t* J0,
                              int64_t N, int gs, InitConsts ic) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < N;
       e += (int64_t)gridDim.x * blockDim.x) {
    const float w = load_w1(W, w_bf16, e);
    const float s = S[e / gs];
    const float u = s != 0.f ? __fdiv_rn(w, s) : 0.f;
    int q = 0;
    for (int k = 0; k + 1 < ic.n_grid; ++k) q += ((double)u > ic.mids[k]) ? 1 : 0;
    double mu[8], mean = 0.0;
    if (ic.relax == GSQ_RELAX_TERNARY) {
      mu[0] = q != 1 ? 1.0 : -1.0;
      mu[1] = (double)(q - 1);
    } else {
      double cq = 0.0;
      for (int k = 0; k < ic.n_grid; ++k) if (k == q) cq = (double)ic.c[k];
      for (int k = 0; k < ic.K; ++k) {
        const double dlt = ic.relax == GSQ_RELAX_SHIFT ? (double)(k - 2) : (double)ic.c[k] - cq;
        mu[k] = -0.5 * dlt * dlt;
        mean += mu[k];
      }
      mean /= (double)ic.K;
      if (ic.relax == GSQ_RELAX_SHIFT) J0[e] = (uint8_t)q;
    }
    float eps[8];
    for (int k = 0; k < 8; ++k) eps[k] = 0.f;
    if (ic.noise) {
      // flat positions (2m, 2m+1) of the chunk's stream form one Box-Muller pair (cos, sin)
      const uint64_t e0 = (uint64_t)e & ~(uint64_t)3;
      const int qq = (int)(e & 3);
      for (int k = 0; k < ic.K; ++k) {
        const int f = qq * ic.K + k;
        const U4 x = noise_words(ic.seed, e0, 0u, 1u, (uint32_t)(f >> 2));
        const int r0 = f & 2;   // the pair's first word within the call
        const double u0 = uniform01(word_of(x, r0)), u1 = uniform01(word_of(x, r0 + 1));
        const double rad = sqrt(-2.0 * log(u0)), ang = 2.0 * M_PI * u1;
        eps[k] = (float)((f & 1) ? rad * sin(ang) : rad * cos(ang));
      }
    }
    for (int k = 0; k < ic.K; ++k)
      L[state_off(e, k, ic.K)] =
          (float)((double)ic.sigma * ((double)eps[k] + (double)ic.alpha * (mu[k] - mean)));
  }
}

// ------------------------------------------------------------------ hardening and packing
// Grid codes: GRID: q = argmax_k l_k (ties to the lowest k); SHIFT: clip(j0 + delta*) with
// delta* the argmax shift; TERNARY: Alg. 2's thresholds, active iff l_m >= 0, positive iff
// l_b >= 0, q = 1 + mask * sign.  Optionally the hard residual R = W - s c[q] (s rounded to
// fp16 in the group layouts) written in the contraction's padded layout, fp32 when
// r_f32 != 0, bf16 otherwise.  Rows and columns as in the forward: four rows per block, four
// consecutive columns per lane (I is a multiple of 16, so a lane's columns share a group).
template <int K, int kMode>
__global__ __launch_bounds__(kBlock) void k_harden(ElemArgs a, int superblock, int r_f32,
                                                   uint8_t* codes, void* Rh) {
  const int lane = threadIdx.x & 63;
  const int64_t col0 = (int64_t)blockIdx.x * kCols + lane * 4;
  const int64_t gpr = a.I / a.gs;
  const bool codes4 = (reinterpret_cast<uintptr_t>(codes) & 3) == 0;
  for (int64_t row = (int64_t)blockIdx.y * 4 + (threadIdx.x >> 6); row < a.rows;
       row += (int64_t)gridDim.y * 4) {
    if (col0 >= a.I) continue;
    const int64_t e0 = row * a.I + col0;
    // every load (logit planes, and W and the scale for the hard residual) is issued before the
    // first comparison and before the byte store of the codes, which the compiler may not move
    // loads across
    float4 lv[K];
#pragma unroll
    for (int k = 0; k < K; ++k) lv[k] = ld_stream(a.L + state_off(e0, k, K));
    float w[4] = {0.f, 0.f, 0.f, 0.f}, s = 0.f;
    if (Rh) {
      s = a.S[row * gpr + col0 / a.gs];
      load_w4(a.W, a.w_bf16, e0, w);
    }
    int q[4] = {0, 0, 0, 0};
    if constexpr (kMode == GSQ_RELAX_TERNARY) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        q[j] = f4get(lv[0], j) >= 0.f ? (f4get(lv[1], j) >= 0.f ? 2 : 0) : 1;
    } else {
      float4 best = lv[0];
#pragma unroll
      for (int k = 1; k < K; ++k) {
        const float4 x = lv[k];
        if (x.x > best.x) { best.x = x.x; q[0] = k; }
        if (x.y > best.y) { best.y = x.y; q[1] = k; }
        if (x.z > best.z) { best.z = x.z; q[2] = k; }
        if (x.w > best.w) { best.w = x.w; q[3] = k; }
      }
      if constexpr (kMode == GSQ_RELAX_SHIFT) {
        const uint32_t j4 = *reinterpret_cast<const uint32_t*>(a.J0 + e0);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int b = (int)((j4 >> (8 * j)) & 0xFFu);
          b = b < a.n_grid ? b : a.n_grid - 1;
          const int c = b + q[j] - 2;
          q[j] = c < 0 ? 0 : (c > a.n_grid - 1 ? a.n_grid - 1 : c);
        }
      }
    }
    if (codes) {
      if (codes4) {
        *reinterpret_cast<uint32_t*>(codes + e0) =
            (uint32_t)q[0] | ((uint32_t)q[1] << 8) | ((uint32_t)q[2] << 16) | ((uint32_t)q[3] << 24);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) codes[e0 + j] = (uint8_t)q[j];
      }
    }
    if (Rh) {
      if (!superblock) s = __half2float(__float2half_rn(s));
      float r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float cq = a.c[0];
        for (int k = 1; k < GSQ_MAX_LEVELS; ++k) if (k == q[j]) cq = a.c[k];
        r[j] = w[j] - s * cq;
      }
      if (r_f32) store_r4<true>(Rh, padded_index(a, row, col0), r);
      else store_r4<false>(Rh, padded_index(a, row, col0), r);
    }
  }
}

// Effective scales: fp16-rounded group scales (flag if one overflows), or the super-block
// scales d * sc unchanged.
__global__ void k_eff_scales(const float* S, float* out, int64_t n, int superblock, int* flag) {
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < n;
       g += (int64_t)gridDim.x * blockDim.x) {
    float s = S[g];
    if (!superblock) s = __half2float(__float2half_rn(s));
    if (!__builtin_isfinite(s)) *flag = 1;
    if (out) out[g] = s;
  }
}

// Plain layout, code section: eight consecutive codes -> b bytes of the LSB-first bitstream.
__global__ void k_pack_codes(const uint8_t* codes, uint8_t* out, int64_t n8, int b) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n8;
       j += (int64_t)gridDim.x * blockDim.x) {
    const uint2 c8 = *reinterpret_cast<const uint2*>(codes + 8 * j);
    uint32_t word = 0;
    for (int q = 0; q < 8; ++q) {
      const uint32_t code = ((q < 4 ? c8.x : c8.y) >> (8 * (q & 3))) & 0xFFu;
      word |= code << (b * q);
    }
    for (int by = 0; by < b; ++by) out[j * b + by] = (uint8_t)(word >> (8 * by));
  }
}

// Base-3 layout, code section: five consecutive codes t_j -> one byte sum_j t_j 3^j (codes past
// the end count as 0).
__global__ void k_pack_base3(const uint8_t* codes, uint8_t* out, int64_t n, int64_t nbytes) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nbytes;
       j += (int64_t)gridDim.x * blockDim.x) {
    uint32_t byte = 0;
    for (int i = 4; i >= 0; --i) {
      const int64_t idx = 5 * j + i;
      byte = 3u * byte + (idx < n ? (uint32_t)codes[idx] : 0u);
    }
    out[j] = (uint8_t)byte;
  }
}

// Plain layout, scale section: fp16 scales, little endian.
__global__ void k_pack_scales(const float* S, uint8_t* out, int64_t n, int* flag) {
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < n;
       g += (int64_t)gridDim.x * blockDim.x) {
    const __half h = __float2half_rn(S[g]);
    if (!__builtin_isfinite(__half2float(h))) *flag = 1;
    const uint16_t bits = __half_as_ushort(h);
    out[2 * g] = (uint8_t)bits;
    out[2 * g + 1] = (uint8_t)(bits >> 8);
  }
}

// Super-block layout: one 110-byte record per 256 weights,
// [fp16 d][16 x 6-bit sc, LSB first][256 x 3-bit codes, LSB first].  A block builds kSbRecs
// consecutive records in LDS (the 3-bit codes of 16 weights fill 6 whole bytes, the 16 sub-block
// scales 12) and writes them out as one contiguous run, so that the code reads (16 bytes per
// lane) and the record writes (4 bytes per lane where `out` allows) are both coalesced.
constexpr int kSbRecs = 64;
constexpr int kSbBytes = 110;

__global__ __launch_bounds__(256) void k_pack_superblock(const uint8_t* __restrict__ codes,
                                                         const uint16_t* __restrict__ D,
                                                         const uint8_t* __restrict__ SC,
                                                         uint8_t* __restrict__ out, int64_t nrec) {
  __shared__ __align__(16) uint8_t buf[kSbRecs * kSbBytes];
  const bool words = (reinterpret_cast<uintptr_t>(out) & 3) == 0;
  for (int64_t r0 = (int64_t)blockIdx.x * kSbRecs; r0 < nrec; r0 += (int64_t)gridDim.x * kSbRecs) {
    const int nr = (int)(nrec - r0 < kSbRecs ? nrec - r0 : kSbRecs);
    // codes: piece p = codes 16 p .. 16 p + 15 of the run -> 6 bytes of record p / 16
    const uint8_t* src = codes + r0 * 256;
    for (int p = threadIdx.x; p < nr * 16; p += blockDim.x) {
      const uint4 c = *reinterpret_cast<const uint4*>(src + 16 * (int64_t)p);
      const uint32_t w4[4] = {c.x, c.y, c.z, c.w};
      uint64_t bits = 0;
#pragma unroll
      for (int q = 0; q < 16; ++q) bits |= (uint64_t)((w4[q >> 2] >> (8 * (q & 3))) & 7u) << (3 * q);
      uint8_t* o = buf + (p >> 4) * kSbBytes + 14 + 6 * (p & 15);
#pragma unroll
      for (int b = 0; b < 6; ++b) o[b] = (uint8_t)(bits >> (8 * b));
    }
    // header of each record: d, then the 96 bits of the 16 sub-block scales
    for (int rec = threadIdx.x; rec < nr; rec += blockDim.x) {
      const int64_t r = r0 + rec;
      uint8_t* o = buf + rec * kSbBytes;
      const uint16_t d = D[r];
      o[0] = (uint8_t)d;
      o[1] = (uint8_t)(d >> 8);
      const uint4 sc = *reinterpret_cast<const uint4*>(SC + 16 * r);
      const uint32_t s4[4] = {sc.x, sc.y, sc.z, sc.w};
      uint64_t lo = 0, hi = 0;   // bits 0..63 and 64..95 of the scale field
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const uint64_t v = (s4[j >> 2] >> (8 * (j & 3))) & 63u;
        const int at = 6 * j;
        if (at < 64) lo |= v << at;
        if (at + 6 > 64) hi |= at >= 64 ? v << (at - 64) : v >> (64 - at);
      }
#pragma unroll
      for (int b = 0; b < 8; ++b) o[2 + b] = (uint8_t)(lo >> (8 * b));
#pragma unroll
      for (int b = 0; b < 4; ++b) o[10 + b] = (uint8_t)(hi >> (8 * b));
    }
    __syncthreads();
    uint8_t* dst = out + r0 * kSbBytes;   // r0 kSbBytes is a multiple of 4
    const int nbytes = nr * kSbBytes;
    const int nw = words ? nbytes / 4 : 0;
    for (int i = threadIdx.x; i < nw; i += blockDim.x)
      reinterpret_cast<uint32_t*>(dst)[i] = reinterpret_cast<const uint32_t*>(buf)[i];
    for (int i = 4 * nw + threadIdx.x; i < nbytes; i += blockDim.x) dst[i] = buf[i];
    __syncthreads();   // buf is refilled by the next run
  }
}

// ------------------------------------------------------------------ state copies
// Between the caller's coordinate-major layout (B, O, I, K) and the blocked planes.
__global__ void k_state_io(float* inter, float* planar, int64_t N, int K, int to_planar) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < N;
       e += (int64_t)gridDim.x * blockDim.x) {
    for (int k = 0; k < K; ++k) {
      if (to_planar) planar[state_off(e, k, K)] = inter[e * K + k];
      else inter[e * K + k] = planar[state_off(e, k, K)];
    }
  }
}

// Padded (B, Opad, Ipad) -> dense (B, O, I); elem_bytes is 2 or 4.
__global__ void k_unpad(const uint8_t* src, uint8_t* dst, int64_t N, int64_t O, int64_t I,
                        int64_t Opad, int64_t Ipad, int elem_bytes) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < N;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = e / I, col = e - row * I;
    const int64_t b = row / O, o = row - b * O;
    const int64_t si = (b * Opad + o) * Ipad + col;
    if (elem_bytes == 4) reinterpret_cast<float*>(dst)[e] = reinterpret_cast<const float*>(src)[si];
    else reinterpret_cast<uint16_t*>(dst)[e] = reinterpret_cast<const uint16_t*>(src)[si];
  }
}

// ------------------------------------------------------------------ noise probe
template <int K, bool kExact, int kKind>
__global__ void k_gumbel(uint64_t seed, int64_t e0, int64_t count, uint32_t t, float* out) {
  for (int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; n < count;
       n += (int64_t)gridDim.x * blockDim.x) {
    float g[K];
    draw_one<K, kExact, kKind>(g, seed, (uint64_t)(e0 + n), t);
    for (int k = 0; k < K; ++k) out[n * K + k] = g[k];
  }
}

dim3 flat_grid(int64_t n, int block = 256) {
  int64_t g = (n + block - 1) / block;
  if (g > 1 << 20) g = 1 << 20;
  if (g < 1) g = 1;
  return dim3((unsigned)g);
}

dim3 row_grid(const Layer& L) {
  const int64_t gx = (L.I + kCols - 1) / kCols;
  int64_t gy = (L.B * L.O + 3) / 4;
  if (gy > 65535) gy = 65535;
  return dim3((unsigned)gx, (unsigned)gy);
}

}  // namespace

int64_t state_floats(const Layer& L) {
  return L.K * ((L.N + kStateBlock - 1) / kStateBlock) * kStateBlock;
}

// ====================================================================== launchers
ElemArgs base_args(const Layer& L) {
  ElemArgs a{};
  a.W = L.W;
  a.G = L.G;
  a.L = L.L; a.M = L.M; a.V = L.V;
  a.S = L.S; a.MS = L.MS; a.VS = L.VS;
  a.flag = L.flag;
  a.loss_part = L.loss_part;
  a.N = L.N;
  a.rows = (int32_t)(L.B * L.O);
  a.O = (int32_t)L.O; a.I = (int32_t)L.I;
  a.Opad = (int32_t)L.Opad; a.Ipad = (int32_t)L.Ipad;
  a.gs = (int32_t)L.gs;
  a.w_bf16 = L.w_bf16;
  a.seed = L.cfg.seed;
  a.J0 = L.J0;
  a.n_grid = L.n_grid;
  for (int k = 0; k < GSQ_MAX_LEVELS; ++k) a.c[k] = k < L.n_grid ? L.cfg.levels[k] : 0.f;
  return a;
}

hipError_t launch_symmetrize_h(const float* Hin, void* Hout, int64_t B, int64_t I, int64_t Ipad,
                               bool bf16, hipStream_t s) {
  dim3 grid((unsigned)(Ipad / 32), (unsigned)(Ipad / 32), (unsigned)B);
  hipLaunchKernelGGL(k_symmetrize, grid, dim3(32, 8), 0, s, Hin, Hout, I, Ipad, bf16 ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_init_scales(const Layer& L, const float* scales_init, float cmax, hipStream_t s) {
  if (L.cfg.layout == GSQ_LAYOUT_SUPERBLOCK) {
    const int64_t nb = L.N / 256;
    hipLaunchKernelGGL(k_init_scales_superblock, flat_grid(nb), dim3(256), 0, s, L.W, L.w_bf16, L.S,
                       L.sb_d, L.sb_sc, nb, cmax);
  } else if (scales_init) {
    return hipMemcpyAsync(L.S, scales_init, L.NG * sizeof(float), hipMemcpyDeviceToDevice, s);
  } else {
    hipLaunchKernelGGL(k_init_scales_group, flat_grid(L.NG), dim3(256), 0, s, L.W, L.w_bf16, L.S,
                       L.NG, (int)L.gs, cmax);
  }
  return hipGetLastError();
}

hipError_t launch_init_logits(const Layer& L, const double* mids, hipStream_t s) {
  InitConsts ic{};
  for (int k = 0; k < GSQ_MAX_LEVELS; ++k) {
    ic.c[k] = k < L.n_grid ? L.cfg.levels[k] : 0.f;
    ic.mids[k] = k + 1 < L.n_grid ? mids[k] : 0.0;
  }
  ic.K = (int)L.K;
  ic.n_grid = L.n_grid;
  ic.relax = L.relax;
  ic.alpha = L.cfg.alpha;
  ic.sigma = L.cfg.sigma_init;
  ic.noise = L.cfg.init_noise;
  ic.seed = L.cfg.seed;
  hipLaunchKernelGGL(k_init_logits, flat_grid(L.N), dim3(256), 0, s, L.W, L.w_bf16, L.S, L.L, L.J0,
                     L.N, (int)L.gs, ic);
  return hipGetLastError();
}

template <int K, int kMode = GSQ_RELAX_GRID>
static hipError_t forward_k(const Layer& L, const ElemArgs& a, hipStream_t s) {
  if (L.bf16) hipLaunchKernelGGL((k_forward<K, false, kMode>), row_grid(L), dim3(kBlock), 0, s, a);
  else hipLaunchKernelGGL((k_forward<K, true, kMode>), row_grid(L), dim3(kBlock), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_forward(const Layer& L, const ElemArgs& a, hipStream_t s) {
  if (L.relax == GSQ_RELAX_SHIFT) return forward_k<GSQ_SHIFT_WINDOW, GSQ_RELAX_SHIFT>(L, a, s);
  if (L.relax == GSQ_RELAX_TERNARY) return forward_k<2, GSQ_RELAX_TERNARY>(L, a, s);
  switch (L.K) {
    case 2: return forward_k<2>(L, a, s);
    case 3: return forward_k<3>(L, a, s);
    case 4: return forward_k<4>(L, a, s);
    case 5: return forward_k<5>(L, a, s);
    case 6: return forward_k<6>(L, a, s);
    case 7: return forward_k<7>(L, a, s);
    default: return forward_k<8>(L, a, s);
  }
}

template <int K, bool kMulti, int kMode, bool kLion>
static void backward_km(const Layer& L, const ElemArgs& a, bool sc, hipStream_t s) {
  const dim3 g = row_grid(L), b(kBlock);
  if (L.bf16) {
    if (sc) hipLaunchKernelGGL((k_backward<K, false, true, kMulti, kMode, kLion>), g, b, 0, s, a);
    else hipLaunchKernelGGL((k_backward<K, false, false, kMulti, kMode, kLion>), g, b, 0, s, a);
  } else {
    if (sc) hipLaunchKernelGGL((k_backward<K, true, true, kMulti, kMode, kLion>), g, b, 0, s, a);
    else hipLaunchKernelGGL((k_backward<K, true, false, kMulti, kMode, kLion>), g, b, 0, s, a);
  }
}

template <int K, int kMode = GSQ_RELAX_GRID>
static hipError_t backward_k(const Layer& L, const ElemArgs& a, bool sc, hipStream_t s) {
  if (a.lion) {
    if (a.samples > 1) backward_km<K, true, kMode, true>(L, a, sc, s);
    else backward_km<K, false, kMode, true>(L, a, sc, s);
  } else {
    if (a.samples > 1) backward_km<K, true, kMode, false>(L, a, sc, s);
    else backward_km<K, false, kMode, false>(L, a, sc, s);
  }
  return hipGetLastError();
}

hipError_t launch_backward(const Layer& L, const ElemArgs& a, bool update_scales, hipStream_t s) {
  if (L.relax == GSQ_RELAX_SHIFT)
    return backward_k<GSQ_SHIFT_WINDOW, GSQ_RELAX_SHIFT>(L, a, update_scales, s);
  if (L.relax == GSQ_RELAX_TERNARY) return backward_k<2, GSQ_RELAX_TERNARY>(L, a, update_scales, s);
  switch (L.K) {
    case 2: return backward_k<2>(L, a, update_scales, s);
    case 3: return backward_k<3>(L, a, update_scales, s);
    case 4: return backward_k<4>(L, a, update_scales, s);
    case 5: return backward_k<5>(L, a, update_scales, s);
    case 6: return backward_k<6>(L, a, update_scales, s);
    case 7: return backward_k<7>(L, a, update_scales, s);
    default: return backward_k<8>(L, a, update_scales, s);
  }
}

template <int K, int kMode = GSQ_RELAX_GRID>
static hipError_t harden_k(const Layer& L, uint8_t* codes, void* Rh, hipStream_t s) {
  hipLaunchKernelGGL((k_harden<K, kMode>), row_grid(L), dim3(kBlock), 0, s, base_args(L),
                     L.cfg.layout == GSQ_LAYOUT_SUPERBLOCK ? 1 : 0, L.bf16 ? 0 : 1, codes, Rh);
  return hipGetLastError();
}

hipError_t launch_harden(const Layer& L, uint8_t* codes, void* Rh, hipStream_t s) {
  if (L.relax == GSQ_RELAX_SHIFT) return harden_k<GSQ_SHIFT_WINDOW, GSQ_RELAX_SHIFT>(L, codes, Rh, s);
  if (L.relax == GSQ_RELAX_TERNARY) return harden_k<2, GSQ_RELAX_TERNARY>(L, codes, Rh, s);
  switch (L.K) {
    case 2: return harden_k<2>(L, codes, Rh, s);
    case 3: return harden_k<3>(L, codes, Rh, s);
    case 4: return harden_k<4>(L, codes, Rh, s);
    case 5: return harden_k<5>(L, codes, Rh, s);
    case 6: return harden_k<6>(L, codes, Rh, s);
    case 7: return harden_k<7>(L, codes, Rh, s);
    default: return harden_k<8>(L, codes, Rh, s);
  }
}

hipError_t launch_eff_scales(const Layer& L, float* out, hipStream_t s) {
  hipLaunchKernelGGL(k_eff_scales, flat_grid(L.NG), dim3(256), 0, s, L.S, out, L.NG,
                     L.cfg.layout == GSQ_LAYOUT_SUPERBLOCK ? 1 : 0, L.flag);
  return hipGetLastError();
}

hipError_t launch_pack(const Layer& L, const uint8_t* codes, uint8_t* out, hipStream_t s) {
  if (L.cfg.layout == GSQ_LAYOUT_SUPERBLOCK) {
    const int64_t nrec = L.N / 256;
    hipLaunchKernelGGL(k_pack_superblock, flat_grid((nrec + kSbRecs - 1) / kSbRecs, 1), dim3(256), 0,
                       s, codes, L.sb_d, L.sb_sc, out, nrec);
    return hipGetLastError();
  }
  int64_t code_bytes;
  if (L.cfg.layout == GSQ_LAYOUT_BASE3) {
    code_bytes = (L.N + 4) / 5;
    hipLaunchKernelGGL(k_pack_base3, flat_grid(code_bytes), dim3(256), 0, s, codes, out, L.N,
                       code_bytes);
  } else {
    const int b = L.n_grid <= 2 ? 1 : L.n_grid <= 4 ? 2 : L.n_grid <= 8 ? 3 : 4;
    const int64_t n8 = L.N / 8;
    code_bytes = L.N * b / 8;
    hipLaunchKernelGGL(k_pack_codes, flat_grid(n8), dim3(256), 0, s, codes, out, n8, b);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(k_pack_scales, flat_grid(L.NG), dim3(256), 0, s, L.S, out + code_bytes, L.NG,
                     L.flag);
  return hipGetLastError();
}

hipError_t launch_state_io(const Layer& L, float* inter, float* planar, bool to_planar,
                           hipStream_t s) {
  hipLaunchKernelGGL(k_state_io, flat_grid(L.N), dim3(256), 0, s, inter, planar, L.N, (int)L.K,
                     to_planar ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_copy_residual(const Layer& L, const void* Rpad, void* out, hipStream_t s) {
  hipLaunchKernelGGL(k_unpad, flat_grid(L.N), dim3(256), 0, s, static_cast<const uint8_t*>(Rpad),
                     static_cast<uint8_t*>(out), L.N, L.O, L.I, L.Opad, L.Ipad, L.bf16 ? 2 : 4);
  return hipGetLastError();
}

hipError_t launch_copy_grad(const Layer& L, const float* Gpad, float* out, hipStream_t s) {
  hipLaunchKernelGGL(k_unpad, flat_grid(L.N), dim3(256), 0, s,
                     reinterpret_cast<const uint8_t*>(Gpad), reinterpret_cast<uint8_t*>(out), L.N,
                     L.O, L.I, L.Opad, L.Ipad, 4);
  return hipGetLastError();
}

template <int K, int kKind = kGumbel>
static hipError_t gumbel_k(const gsq_config& cfg, int64_t e0, int64_t count, int64_t t, float* out,
                           hipStream_t s) {
  if (cfg.precision == GSQ_PREC_BF16)
    hipLaunchKernelGGL((k_gumbel<K, false, kKind>), flat_grid(count), dim3(256), 0, s, cfg.seed, e0,
                       count, (uint32_t)t, out);
  else
    hipLaunchKernelGGL((k_gumbel<K, true, kKind>), flat_grid(count), dim3(256), 0, s, cfg.seed, e0,
                       count, (uint32_t)t, out);
  return hipGetLastError();
}

hipError_t launch_gumbel(const gsq_config& cfg, int64_t e0, int64_t count, int64_t t, float* out,
                         hipStream_t s) {
  if (cfg.relaxation == GSQ_RELAX_TERNARY) return gumbel_k<2, kLogistic>(cfg, e0, count, t, out, s);
  const int z = cfg.relaxation == GSQ_RELAX_SHIFT ? GSQ_SHIFT_WINDOW : cfg.n_levels;
  switch (z) {
    case 2: return gumbel_k<2>(cfg, e0, count, t, out, s);
    case 3: return gumbel_k<3>(cfg, e0, count, t, out, s);
    case 4: return gumbel_k<4>(cfg, e0, count, t, out, s);
    case 5: return gumbel_k<5>(cfg, e0, count, t, out, s);
    case 6: return gumbel_k<6>(cfg, e0, count, t, out, s);
    case 7: return gumbel_k<7>(cfg, e0, count, t, out, s);
    default: return gumbel_k<8>(cfg, e0, count, t, out, s);
  }
}

}  // namespace gsq
