// Host side of the C ABI in gsq.h: validation, buffer ownership and launch order.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "gsq_internal.h"

namespace {

thread_local std::string g_err;

gsq_status fail(gsq_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

gsq_status hip_fail(hipError_t e, const char* what) {
  return fail(GSQ_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define GSQ_HIP(call)                                  \
  do {                                                 \
    hipError_t e_ = (call);                            \
    if (e_ != hipSuccess) return hip_fail(e_, #call);  \
  } while (0)

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

int code_bits(int n) { return n <= 2 ? 1 : n <= 4 ? 2 : n <= 8 ? 3 : 4; }

int logits_per_coord(const gsq_config& c) {
  return c.relaxation == GSQ_RELAX_SHIFT ? GSQ_SHIFT_WINDOW
         : c.relaxation == GSQ_RELAX_TERNARY ? 2 : c.n_levels;
}

gsq_status validate_config(const gsq_config* c) {
  if (!c) return fail(GSQ_EINVAL, "config is NULL");
  if (c->batch < 1 || c->out_features < 1 || c->in_features < 1)
    return fail(GSQ_EINVAL, "batch, out_features and in_features must be >= 1");
  if (c->relaxation != GSQ_RELAX_GRID && c->relaxation != GSQ_RELAX_SHIFT &&
      c->relaxation != GSQ_RELAX_TERNARY)
    return fail(GSQ_EINVAL, "unknown relaxation %d", c->relaxation);
  const int nmax = c->relaxation == GSQ_RELAX_SHIFT ? GSQ_MAX_LEVELS : 8;
  if (c->n_levels < 2 || c->n_levels > nmax)
    return fail(GSQ_EINVAL, "n_levels must be in [2, %d] for this relaxation, got %d", nmax,
                c->n_levels);
  if (c->relaxation == GSQ_RELAX_TERNARY &&
      !(c->n_levels == 3 && c->levels[0] == -1.f && c->levels[1] == 0.f && c->levels[2] == 1.f))
    return fail(GSQ_EINVAL, "TERNARY needs the levels {-1, 0, 1}");
  float cmax = 0.f;
  for (int k = 0; k < c->n_levels; ++k) {
    if (!std::isfinite(c->levels[k])) return fail(GSQ_EINVAL, "level %d is not finite", k);
    if (k && !(c->levels[k] > c->levels[k - 1]))
      return fail(GSQ_EINVAL, "levels must be strictly increasing");
    cmax = std::fmax(cmax, std::fabs(c->levels[k]));
  }
  if (cmax == 0.f) return fail(GSQ_EINVAL, "levels are all zero");
  if (c->layout == GSQ_LAYOUT_GROUP || c->layout == GSQ_LAYOUT_BASE3) {
    if (c->layout == GSQ_LAYOUT_BASE3 && c->n_levels != 3)
      return fail(GSQ_EINVAL, "BASE3 stores 3-level codes, got n_levels %d", c->n_levels);
    const int gs = c->group_size;
    if (gs != 16 && gs != 32 && gs != 64 && gs != 128 && gs != 256)
      return fail(GSQ_EINVAL, "group_size must be 16, 32, 64, 128 or 256, got %d", gs);
    if (c->in_features % gs) return fail(GSQ_EINVAL, "in_features must be a multiple of group_size");
  } else if (c->layout == GSQ_LAYOUT_SUPERBLOCK) {
    if (c->in_features % 256) return fail(GSQ_EINVAL, "SUPERBLOCK needs in_features % 256 == 0");
    if (c->n_levels > 8) return fail(GSQ_EINVAL, "SUPERBLOCK stores 3-bit codes (n_levels <= 8)");
  } else {
    return fail(GSQ_EINVAL, "unknown layout %d", c->layout);
  }
  if (c->precision != GSQ_PREC_FP32 && c->precision != GSQ_PREC_BF16)
    return fail(GSQ_EINVAL, "unknown precision %d", c->precision);
  if (!std::isfinite(c->alpha) || !std::isfinite(c->sigma_init))
    return fail(GSQ_EINVAL, "alpha and sigma_init must be finite");
  const int64_t rows = (int64_t)c->batch * c->out_features;
  if (rows > (int64_t)INT32_MAX / 2 || c->in_features > (1 << 24))
    return fail(GSQ_EINVAL, "layer too large for this library's indexing");
  return GSQ_OK;
}

void free_layer(gsq::Layer* L) {
  if (!L) return;
  for (auto& p : L->pending) {
    (void)hipEventDestroy(p.second.first);
    (void)hipEventDestroy(p.second.second);
  }
  for (hipEvent_t e : L->event_pool) (void)hipEventDestroy(e);
  void* bufs[] = {L->W, L->H, L->L, L->M, L->V, L->S, L->MS, L->VS, L->R[0], L->R[1],
                  L->G, L->partials, L->loss_part, L->loss_stage, L->loss_tickets, L->split_ws,
                  L->flag, L->sb_d, L->sb_sc, L->codes,
                  L->J0};
  for (void* p : bufs)
    if (p) (void)hipFree(p);
  delete L;
}

template <typename T>
bool alloc(T** p, size_t bytes) {
  void* q = nullptr;
  if (hipMalloc(&q, bytes == 0 ? 1 : bytes) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  *p = static_cast<T*>(q);
  return true;
}

// Event pair around one launch when timing is on (gsq_timing).
constexpr size_t kMaxPending = 8192;

hipError_t harvest(gsq::Layer& L) {
  size_t done = 0;
  hipError_t e = hipSuccess;
  for (; done < L.pending.size(); ++done) {
    auto& p = L.pending[done];
    e = hipEventSynchronize(p.second.second);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.second.first, p.second.second);
    if (e != hipSuccess) break;
    L.timed_ms[p.first] += ms;
    L.timed_launches[p.first] += 1;
    L.event_pool.push_back(p.second.first);
    L.event_pool.push_back(p.second.second);
  }
  // only the pairs that were read go back to the pool
  L.pending.erase(L.pending.begin(), L.pending.begin() + done);
  return e;
}

hipError_t take_event(gsq::Layer& L, hipEvent_t* e) {
  if (!L.event_pool.empty()) {
    *e = L.event_pool.back();
    L.event_pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(e);
}

template <class F>
hipError_t timed(gsq::Layer& L, int kind, hipStream_t s, F&& launch) {
  if (!L.timing) return launch();
  if (L.pending.size() >= kMaxPending) {
    hipError_t e = harvest(L);
    if (e != hipSuccess) return e;
  }
  hipEvent_t e0, e1;
  hipError_t e = take_event(L, &e0);
  if (e == hipSuccess) e = take_event(L, &e1);
  if (e == hipSuccess) e = hipEventRecord(e0, s);
  if (e == hipSuccess) e = launch();
  if (e == hipSuccess) e = hipEventRecord(e1, s);
  if (e == hipSuccess) L.pending.push_back({kind, {e0, e1}});
  return e;
}

gsq_status check_flag(gsq::Layer* h, hipStream_t s) {
  int flag = 0;
  GSQ_HIP(hipMemcpyAsync(&flag, h->flag, sizeof(int), hipMemcpyDeviceToHost, s));
  GSQ_HIP(hipStreamSynchronize(s));
  if (flag) return fail(GSQ_ENONFINITE, "a loss, gradient, parameter or fp16 scale was not finite");
  return GSQ_OK;
}

// ---- scratch of gsq_step_static: a file-scope device array instead of the handle's buffers.
// It holds the loss reduction's row partials, chunk sums and per-layer tickets.  Each GPU holds
// its own copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device (taken once per device, at the first
// gsq_layer_init on it).  Every gsq_step_static call on a GPU shares that GPU's copy.
constexpr size_t kStaticPartials = (size_t)4 << 20;   // row partials (fp64): 32 MiB
constexpr size_t kStaticStage = (size_t)1 << 16;      // chunk sums (fp64): 512 KiB
constexpr size_t kStaticTickets = (size_t)1 << 16;    // one per layer (u32): 256 KiB
constexpr size_t kStaticBytes = (kStaticPartials + kStaticStage) * 8 + kStaticTickets * 4;
static __device__ __align__(256) unsigned char scratch[kStaticBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {nullptr};

// Address of this device's scratch (device `dev` current), set up on first use: the ticket
// region is cleared, since the reduction leaves tickets at zero but needs them zero on entry.
// Synchronises `stream` the first time only.
hipError_t static_scratch(int dev, hipStream_t stream, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    unsigned char* base = static_cast<unsigned char*>(ptr);
    e = hipMemsetAsync(base + (kStaticPartials + kStaticStage) * 8, 0, kStaticTickets * 4, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

struct gsq_layer : gsq::Layer {};

extern "C" {

const char* gsq_last_error(void) { return g_err.c_str(); }

size_t gsq_packed_size(const gsq_config* cfg) {
  if (validate_config(cfg) != GSQ_OK) return 0;
  const int64_t n = (int64_t)cfg->batch * cfg->out_features * cfg->in_features;
  if (cfg->layout == GSQ_LAYOUT_SUPERBLOCK) return (size_t)(n / 256 * 110);
  const int64_t scales = 2 * (n / cfg->group_size);
  if (cfg->layout == GSQ_LAYOUT_BASE3) return (size_t)((n + 4) / 5 + scales);
  return (size_t)(n * code_bits(cfg->n_levels) / 8 + scales);
}

gsq_status gsq_layer_init(const gsq_config* cfg, const void* W, int32_t w_dtype, const float* H,
                          const float* scales_init, hipStream_t stream, gsq_layer** out) {
  g_err.clear();
  if (!out) return fail(GSQ_EINVAL, "out is NULL");
  *out = nullptr;
  gsq_status st = validate_config(cfg);
  if (st != GSQ_OK) return st;
  if (!W || !H) return fail(GSQ_EINVAL, "W and H must be device pointers");
  if (w_dtype != GSQ_DT_FP32 && w_dtype != GSQ_DT_BF16) return fail(GSQ_EINVAL, "unknown w_dtype");
  if (scales_init && cfg->layout == GSQ_LAYOUT_SUPERBLOCK)
    return fail(GSQ_EINVAL, "scales_init must be NULL for SUPERBLOCK");

  gsq_layer* h = new (std::nothrow) gsq_layer();
  if (!h) return fail(GSQ_ENOMEM, "host allocation failed");
  gsq::Layer& L = *h;
  L.cfg = *cfg;
  L.B = cfg->batch; L.O = cfg->out_features; L.I = cfg->in_features;
  L.K = logits_per_coord(*cfg);
  L.n_grid = cfg->n_levels;
  L.relax = cfg->relaxation;
  L.gs = cfg->layout == GSQ_LAYOUT_SUPERBLOCK ? 16 : cfg->group_size;
  L.Opad = round_up(L.O, gsq::kTileM);
  L.Ipad = round_up(L.I, gsq::kPadK);
  L.N = L.B * L.O * L.I;
  L.NG = L.N / L.gs;
  L.bf16 = cfg->precision == GSQ_PREC_BF16;
  L.w_bf16 = w_dtype == GSQ_DT_BF16 ? 1 : 0;
  const size_t relem = L.bf16 ? 2 : 4;
  const size_t npad = (size_t)(L.B * L.Opad * L.Ipad);
  L.tiles_per_batch = gsq::contract_tiles_per_batch(L);
  L.loss_cols = (L.I + 255) / 256;
  {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) == hipSuccess) {
      L.device = dev;
      if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
        gsq::plan_contract_split(L, ncu);
    }
    (void)hipGetLastError();
  }
  if (L.bf16) {
    // the contraction's LDS ring exceeds the default limit (set on the current device)
    const hipError_t e = gsq::prepare_contract_kernel();
    if (e != hipSuccess) {
      delete h;
      return hip_fail(e, "hipFuncSetAttribute");
    }
  }
  bool ok = alloc(&L.W, L.N * (L.w_bf16 ? 2 : 4)) &&
            alloc(&L.H, (size_t)(L.B * L.Ipad * L.Ipad) * relem) &&
            alloc(&L.L, gsq::state_floats(L) * 4) && alloc(&L.M, gsq::state_floats(L) * 4) &&
            alloc(&L.V, gsq::state_floats(L) * 4) &&
            alloc(&L.S, L.NG * 4) && alloc(&L.MS, L.NG * 4) && alloc(&L.VS, L.NG * 4) &&
            alloc(&L.R[0], npad * relem) && alloc(&L.R[1], npad * relem) &&
            alloc(&L.G, npad * 4) && alloc(&L.partials, (size_t)(L.B * L.tiles_per_batch) * 8) &&
            alloc(&L.loss_part, (size_t)(L.B * L.O * L.loss_cols) * 8) &&
            alloc(&L.loss_stage, (size_t)gsq::loss_stage_size(L) * 8) &&
            alloc(&L.loss_tickets, (size_t)L.B * sizeof(unsigned)) &&
            alloc(&L.flag, sizeof(int)) && alloc(&L.codes, (size_t)L.N);
  if (ok && cfg->layout == GSQ_LAYOUT_SUPERBLOCK)
    ok = alloc(&L.sb_d, (L.N / 256) * 2) && alloc(&L.sb_sc, L.N / 16);
  if (ok && cfg->relaxation == GSQ_RELAX_SHIFT) ok = alloc(&L.J0, (size_t)L.N);
  if (ok && L.split_parts > 1) ok = alloc(&L.split_ws, (size_t)gsq::contract_split_ws_floats(L) * 4);
  if (!ok) {
    free_layer(h);
    return fail(GSQ_ENOMEM, "device allocation failed for a %lld x %lld x %lld layer",
                (long long)L.B, (long long)L.O, (long long)L.I);
  }
  auto run = [&]() -> gsq_status {
    GSQ_HIP(hipMemcpyAsync(L.W, W, L.N * (L.w_bf16 ? 2 : 4), hipMemcpyDeviceToDevice, stream));
    GSQ_HIP(timed(L, GSQ_KERNEL_INIT, stream, [&] { return gsq::launch_symmetrize_h(H, L.H, L.B, L.I, L.Ipad, L.bf16, stream); }));
    GSQ_HIP(hipMemsetAsync(L.R[0], 0, npad * relem, stream));   // padding stays zero
    GSQ_HIP(hipMemsetAsync(L.R[1], 0, npad * relem, stream));
    GSQ_HIP(hipMemsetAsync(L.M, 0, gsq::state_floats(L) * 4, stream));
    GSQ_HIP(hipMemsetAsync(L.V, 0, gsq::state_floats(L) * 4, stream));
    GSQ_HIP(hipMemsetAsync(L.MS, 0, L.NG * 4, stream));
    GSQ_HIP(hipMemsetAsync(L.VS, 0, L.NG * 4, stream));
    GSQ_HIP(hipMemsetAsync(L.flag, 0, sizeof(int), stream));
    GSQ_HIP(hipMemsetAsync(L.loss_tickets, 0, (size_t)L.B * sizeof(unsigned), stream));
    float cmax = 0.f;
    for (int k = 0; k < L.n_grid; ++k) cmax = std::fmax(cmax, std::fabs(cfg->levels[k]));
    GSQ_HIP(timed(L, GSQ_KERNEL_INIT, stream, [&] { return gsq::launch_init_scales(L, scales_init, cmax, stream); }));
    double mids[GSQ_MAX_LEVELS] = {0};
    for (int k = 0; k + 1 < L.n_grid; ++k)
      mids[k] = 0.5 * ((double)cfg->levels[k] + (double)cfg->levels[k + 1]);
    GSQ_HIP(timed(L, GSQ_KERNEL_INIT, stream, [&] { return gsq::launch_init_logits(L, mids, stream); }));
    return GSQ_OK;
  };
  st = run();
  if (st != GSQ_OK) {
    (void)hipStreamSynchronize(stream);
    free_layer(h);
    return st;
  }
  {
    // gsq_step_static's scratch on this device (once per device); a failure here only disables
    // that entry point, which then reports it
    void* unused = nullptr;
    if (static_scratch(L.device, stream, &unused) != hipSuccess) (void)hipGetLastError();
  }
  *out = h;
  return GSQ_OK;
}

// Room for M per-sample gradients (a step asking for more samples than any before it); the
// old buffer is released after the device is idle.
static gsq_status grow_sample_slots(gsq::Layer& L, int M) {
  const size_t npad = (size_t)(L.B * L.Opad * L.Ipad);
  float* G = nullptr;
  if (!alloc(&G, (size_t)M * npad * 4)) return fail(GSQ_ENOMEM, "no room for %d samples", M);
  const hipError_t e = hipDeviceSynchronize();   // no launch on any stream still reads the old one
  if (e != hipSuccess) {
    (void)hipFree(G);
    return hip_fail(e, "hipDeviceSynchronize");
  }
  (void)hipFree(L.G);
  L.G = G;
  L.sample_slots = M;
  L.last = -1;
  return GSQ_OK;
}

static gsq_status validate_params(const gsq_layer* h, const gsq_step_params* p) {
  if (!p) return fail(GSQ_EINVAL, "params is NULL");
  if (!(std::isfinite(p->tau) && p->tau > 0.f)) return fail(GSQ_EINVAL, "tau must be finite and > 0");
  if (!std::isfinite(p->kappa)) return fail(GSQ_EINVAL, "kappa must be finite");
  if (!(std::isfinite(p->lr_logits) && p->lr_logits >= 0.f && std::isfinite(p->lr_scales) &&
        p->lr_scales >= 0.f))
    return fail(GSQ_EINVAL, "learning rates must be finite and >= 0");
  if (!(p->beta1 >= 0.f && p->beta1 < 1.f && p->beta2 >= 0.f && p->beta2 < 1.f))
    return fail(GSQ_EINVAL, "beta1 and beta2 must lie in [0, 1)");
  if (!(std::isfinite(p->eps) && p->eps > 0.f)) return fail(GSQ_EINVAL, "eps must be finite and > 0");
  if (!(std::isfinite(p->tau_next) && p->tau_next >= 0.f && std::isfinite(p->kappa_next)))
    return fail(GSQ_EINVAL, "tau_next must be finite and >= 0, kappa_next finite");
  if (p->optimizer != GSQ_OPT_ADAM && p->optimizer != GSQ_OPT_LION)
    return fail(GSQ_EINVAL, "unknown optimizer %d", p->optimizer);
  if (!(std::isfinite(p->weight_decay) && p->weight_decay >= 0.f))
    return fail(GSQ_EINVAL, "weight_decay must be finite and >= 0");
  if (p->samples < 0 || p->samples > GSQ_MAX_SAMPLES)
    return fail(GSQ_EINVAL, "samples must be in [0, %d]", GSQ_MAX_SAMPLES);
  if (h->cfg.layout == GSQ_LAYOUT_SUPERBLOCK && p->lr_scales != 0.f)
    return fail(GSQ_EUNSUPPORTED, "SUPERBLOCK scales stay on their 6-bit grid: lr_scales must be 0");
  return GSQ_OK;
}

// Buffers of the loss reduction of one step: the handle's own, or gsq_step_static's scratch.
struct LossBuffers {
  double* part;
  double* stage;
  unsigned* tickets;
};

// The body of gsq_step and gsq_step_static, after validation (M sample slots exist).
static gsq_status step_impl(gsq::Layer& L, const gsq_step_params* p, float* loss_out,
                            const LossBuffers& lb, hipStream_t stream) {
  const int M = p->samples > 1 ? p->samples : 1;
  gsq::ElemArgs a = gsq::base_args(L);
  a.loss_part = lb.part;
  a.t = (uint32_t)L.t;
  a.noise = p->gumbel_noise ? 1 : 0;
  a.kappa = p->kappa;
  a.inv_tau = 1.0f / p->tau;
  a.inv_tau_d = 1.0 / (double)p->tau;

  const bool have = L.r_valid && L.r_t == L.t && L.r_tau == p->tau && L.r_kappa == p->kappa &&
                    L.r_noise == a.noise;
  // until this step has been enqueued completely, no prepared sample or intermediate is claimed
  L.r_valid = false;
  L.last = -1;
  const int use = L.cur;
  a.Rout = L.R[use];
  for (int smp = 0; smp < M; ++smp) {
    // sample 0 may have been drawn by the previous step; later samples reuse the buffer
    if (smp > 0 || !have) {
      a.sample = smp;
      GSQ_HIP(timed(L, GSQ_KERNEL_FORWARD, stream, [&] { return gsq::launch_forward(L, a, stream); }));
    }
    GSQ_HIP(timed(L, GSQ_KERNEL_CONTRACT, stream, [&] { return gsq::launch_contract(L, L.R[use], false, smp, stream); }));
  }
  a.want_loss = loss_out ? 1 : 0;   // the backward sums the loss terms of every sample
  a.sample = 0;
  a.samples = M;
  a.g_stride = L.B * L.Opad * L.Ipad;

  const double n = (double)(L.t + 1);
  const double bc1 = 1.0 - std::pow((double)p->beta1, n);
  const double bc2 = 1.0 - std::pow((double)p->beta2, n);
  a.lion = p->optimizer == GSQ_OPT_LION ? 1 : 0;
  a.wd = p->weight_decay;
  a.lr = p->lr_logits;
  a.lr_s = p->lr_scales;
  a.b1 = p->beta1; a.b2 = p->beta2; a.eps = p->eps;
  a.step_l_d = (double)p->lr_logits / bc1;
  a.step_s_d = (double)p->lr_scales / bc1;
  a.rbc2_d = 1.0 / std::sqrt(bc2);
  a.step_l = (float)a.step_l_d;
  a.step_s = (float)a.step_s_d;
  a.rbc2 = (float)a.rbc2_d;
  a.fuse = p->tau_next > 0.f ? 1 : 0;
  a.t_next = (uint32_t)(L.t + 1);
  a.kappa_n = p->kappa_next;
  a.inv_tau_n = a.fuse ? 1.0f / p->tau_next : 0.f;
  a.inv_tau_n_d = a.fuse ? 1.0 / (double)p->tau_next : 0.0;
  a.Rout = L.R[1 - use];
  GSQ_HIP(timed(L, GSQ_KERNEL_BACKWARD, stream, [&] { return gsq::launch_backward(L, a, p->lr_scales > 0.f, stream); }));
  if (loss_out)
    GSQ_HIP(timed(L, GSQ_KERNEL_REDUCE, stream, [&] {
      return gsq::launch_reduce_loss(L, lb.part, lb.stage, lb.tickets, loss_out, true, 1.0 / M, stream);
    }));

  L.last = use;
  L.last_sample = M - 1;
  L.t += 1;
  if (a.fuse) {
    L.cur = 1 - use;
    L.r_valid = true;
    L.r_t = L.t;
    L.r_tau = p->tau_next;
    L.r_kappa = p->kappa_next;
    L.r_noise = a.noise;
  } else {
    L.cur = 1 - use;       // keep the last step's residual readable
    L.r_valid = false;
  }
  return GSQ_OK;
}

gsq_status gsq_step(gsq_layer* h, const gsq_step_params* p, float* loss_out, hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  gsq_status st = validate_params(h, p);
  if (st != GSQ_OK) return st;
  gsq::Layer& L = *h;
  if (L.t >= (int64_t)UINT32_MAX) return fail(GSQ_EINVAL, "step counter exhausted");
  // grow the per-sample buffers before any launch argument captures their addresses
  const int M = p->samples > 1 ? p->samples : 1;
  if (M > L.sample_slots) {
    gsq_status st2 = grow_sample_slots(L, M);
    if (st2 != GSQ_OK) return st2;
  }
  return step_impl(L, p, loss_out, LossBuffers{L.loss_part, L.loss_stage, L.loss_tickets}, stream);
}

gsq_status gsq_step_static(gsq_layer* h, const gsq_step_params* p, float* loss_out,
                           hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  gsq_status st = validate_params(h, p);
  if (st != GSQ_OK) return st;
  gsq::Layer& L = *h;
  if (L.t >= (int64_t)UINT32_MAX) return fail(GSQ_EINVAL, "step counter exhausted");
  const int M = p->samples > 1 ? p->samples : 1;
  if (M > L.sample_slots)
    return fail(GSQ_EINVAL,
                "gsq_step_static allocates nothing: %d samples need per-sample buffers this handle "
                "does not have yet (it has %d; a gsq_step with that many samples creates them)",
                M, L.sample_slots);
  LossBuffers lb{nullptr, nullptr, nullptr};
  if (loss_out) {
    const int64_t np = gsq::loss_row_partials(L), ns = gsq::loss_row_stage(L);
    if (np > (int64_t)kStaticPartials || ns > (int64_t)kStaticStage || L.B > (int64_t)kStaticTickets)
      return fail(GSQ_EINVAL,
                  "gsq_step_static's scratch holds %zu loss partials, %zu chunk sums and %zu layers; "
                  "this layer needs %lld, %lld and %lld (use gsq_step)",
                  kStaticPartials, kStaticStage, kStaticTickets, (long long)np, (long long)ns,
                  (long long)L.B);
    int dev = -1;
    GSQ_HIP(hipGetDevice(&dev));
    if (dev != L.device)
      return fail(GSQ_EINVAL, "the handle was created on device %d, device %d is current", L.device, dev);
    void* base = nullptr;
    {
      std::lock_guard<std::mutex> lock(g_scratch_mu);
      base = dev >= 0 && dev < kMaxDevices ? g_scratch_ptr[dev] : nullptr;
    }
    if (!base) return fail(GSQ_EHIP, "the static scratch of device %d could not be set up", dev);
    unsigned char* b8 = static_cast<unsigned char*>(base);
    lb.part = reinterpret_cast<double*>(b8);
    lb.stage = reinterpret_cast<double*>(b8 + kStaticPartials * 8);
    lb.tickets = reinterpret_cast<unsigned*>(b8 + (kStaticPartials + kStaticStage) * 8);
  }
  return step_impl(L, p, loss_out, lb, stream);
}

gsq_status gsq_harden(gsq_layer* h, uint8_t* codes, float* scales, float* hard_loss_out,
                      hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  gsq::Layer& L = *h;
  void* Rh = nullptr;
  if (hard_loss_out) {
    // the hard residual goes to the buffer that does not hold the last step's residual
    const int buf = L.last >= 0 ? 1 - L.last : L.cur;
    Rh = L.R[buf];
    L.r_valid = false;
  }
  GSQ_HIP(timed(L, GSQ_KERNEL_HARDEN, stream, [&] { return gsq::launch_harden(L, codes ? codes : L.codes, Rh, stream); }));
  GSQ_HIP(timed(L, GSQ_KERNEL_HARDEN, stream, [&] { return gsq::launch_eff_scales(L, scales, stream); }));
  if (hard_loss_out) {
    GSQ_HIP(timed(L, GSQ_KERNEL_CONTRACT, stream, [&] { return gsq::launch_contract(L, Rh, true, 0, stream); }));
    GSQ_HIP(timed(L, GSQ_KERNEL_REDUCE, stream, [&] { return gsq::launch_reduce_loss(L, hard_loss_out, false, 1.0, stream); }));
    L.last = -1;   // G now belongs to the hard residual
    L.last_sample = 0;
  }
  return check_flag(h, stream);
}

gsq_status gsq_pack(gsq_layer* h, void* packed, size_t packed_bytes, hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  if (!packed) return fail(GSQ_EINVAL, "packed is NULL");
  const size_t need = gsq_packed_size(&h->cfg);
  if (packed_bytes < need)
    return fail(GSQ_EINVAL, "packed buffer has %zu bytes, needs %zu", packed_bytes, need);
  gsq::Layer& L = *h;
  GSQ_HIP(timed(L, GSQ_KERNEL_HARDEN, stream, [&] { return gsq::launch_harden(L, L.codes, nullptr, stream); }));
  GSQ_HIP(timed(L, GSQ_KERNEL_PACK, stream, [&] { return gsq::launch_pack(L, L.codes, static_cast<uint8_t*>(packed), stream); }));
  return check_flag(h, stream);
}

gsq_status gsq_get_state(gsq_layer* h, float* logits, float* m, float* v, float* scales, float* m_s,
                         float* v_s, uint8_t* base, int64_t* t, hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  gsq::Layer& L = *h;
  if (base && !L.J0) return fail(GSQ_EINVAL, "base indices exist only for the SHIFT relaxation");
  if (base) GSQ_HIP(hipMemcpyAsync(base, L.J0, (size_t)L.N, hipMemcpyDeviceToDevice, stream));
  if (logits) GSQ_HIP(gsq::launch_state_io(L, logits, L.L, false, stream));
  if (m) GSQ_HIP(gsq::launch_state_io(L, m, L.M, false, stream));
  if (v) GSQ_HIP(gsq::launch_state_io(L, v, L.V, false, stream));
  const size_t sb = L.NG * 4;
  if (scales) GSQ_HIP(hipMemcpyAsync(scales, L.S, sb, hipMemcpyDeviceToDevice, stream));
  if (m_s) GSQ_HIP(hipMemcpyAsync(m_s, L.MS, sb, hipMemcpyDeviceToDevice, stream));
  if (v_s) GSQ_HIP(hipMemcpyAsync(v_s, L.VS, sb, hipMemcpyDeviceToDevice, stream));
  if (t) *t = L.t;
  return check_flag(h, stream);
}

gsq_status gsq_set_state(gsq_layer* h, const float* logits, const float* m, const float* v,
                         const float* scales, const float* m_s, const float* v_s,
                         const uint8_t* base, int64_t t, hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  if (t < 0 || t >= (int64_t)UINT32_MAX) return fail(GSQ_EINVAL, "t out of range");
  gsq::Layer& L = *h;
  if (base && !L.J0) return fail(GSQ_EINVAL, "base indices exist only for the SHIFT relaxation");
  if (scales && L.cfg.layout == GSQ_LAYOUT_SUPERBLOCK)
    return fail(GSQ_EUNSUPPORTED, "SUPERBLOCK scales are fixed by their 6-bit encoding");
  if (base) GSQ_HIP(hipMemcpyAsync(L.J0, base, (size_t)L.N, hipMemcpyDeviceToDevice, stream));
  if (logits) GSQ_HIP(gsq::launch_state_io(L, const_cast<float*>(logits), L.L, true, stream));
  if (m) GSQ_HIP(gsq::launch_state_io(L, const_cast<float*>(m), L.M, true, stream));
  if (v) GSQ_HIP(gsq::launch_state_io(L, const_cast<float*>(v), L.V, true, stream));
  const size_t sb = L.NG * 4;
  if (scales) GSQ_HIP(hipMemcpyAsync(L.S, scales, sb, hipMemcpyDeviceToDevice, stream));
  if (m_s) GSQ_HIP(hipMemcpyAsync(L.MS, m_s, sb, hipMemcpyDeviceToDevice, stream));
  if (v_s) GSQ_HIP(hipMemcpyAsync(L.VS, v_s, sb, hipMemcpyDeviceToDevice, stream));
  L.t = t;
  L.r_valid = false;
  L.last = -1;
  return GSQ_OK;
}

gsq_status gsq_get_intermediates(gsq_layer* h, void* residual, float* grad, hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  gsq::Layer& L = *h;
  if (L.last < 0) return fail(GSQ_EINVAL, "no step has run since init, set_state or harden");
  if (residual) GSQ_HIP(gsq::launch_copy_residual(L, L.R[L.last], residual, stream));
  if (grad)
    GSQ_HIP(gsq::launch_copy_grad(L, L.G + (int64_t)L.last_sample * L.B * L.Opad * L.Ipad, grad, stream));
  return GSQ_OK;
}

gsq_status gsq_gumbel(const gsq_config* cfg, int64_t e0, int64_t count, int64_t t, float* g_out,
                      hipStream_t stream) {
  g_err.clear();
  gsq_status st = validate_config(cfg);
  if (st != GSQ_OK) return st;
  if (e0 < 0 || count < 0 || t < 0 || t >= (int64_t)UINT32_MAX)
    return fail(GSQ_EINVAL, "e0, count and t must be >= 0 (t < 2^32)");
  if (count == 0) return GSQ_OK;
  if (!g_out) return fail(GSQ_EINVAL, "g_out is NULL");
  GSQ_HIP(gsq::launch_gumbel(*cfg, e0, count, t, g_out, stream));
  return GSQ_OK;
}

gsq_status gsq_timing(gsq_layer* h, int32_t enable) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  h->timing = enable != 0;
  return GSQ_OK;
}

gsq_status gsq_timing_read(gsq_layer* h, double* ms, int64_t* launches, int32_t reset,
                           hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  GSQ_HIP(hipStreamSynchronize(stream));
  GSQ_HIP(harvest(*h));
  for (int k = 0; k < GSQ_NUM_KERNELS; ++k) {
    if (ms) ms[k] = h->timed_ms[k];
    if (launches) launches[k] = h->timed_launches[k];
    if (reset) {
      h->timed_ms[k] = 0.0;
      h->timed_launches[k] = 0;
    }
  }
  return GSQ_OK;
}

gsq_status gsq_check(gsq_layer* h, hipStream_t stream) {
  g_err.clear();
  if (!h) return fail(GSQ_EINVAL, "handle is NULL");
  return check_flag(h, stream);
}

gsq_status gsq_layer_destroy(gsq_layer* h) {
  if (!h) return GSQ_OK;
  (void)hipDeviceSynchronize();
  free_layer(h);
  return GSQ_OK;
}

}  // extern "C"
