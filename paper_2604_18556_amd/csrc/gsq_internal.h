// Internal declarations shared by the host API and the kernel launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>
#include <vector>

#include "gsq.h"

namespace gsq {

constexpr int kTileM = 256;   // contraction tile (rows of R / G)
constexpr int kTileN = 256;   // contraction tile (columns of G = rows of H)
constexpr int kPadK = 256;    // padding of the inner dimension (H is padded with zeros)
// Layout of the logits and of each optimiser moment: blocks of kStateBlock consecutive
// coordinates, the K planes of a block side by side (plane k of block j starts at float
// (j K + k) kStateBlock).  The arrays hold whole blocks.
constexpr int64_t kStateBlock = 16384;

// Everything an elementwise kernel needs, passed by value.
struct ElemArgs {
  const void* W;        // B*O*I, fp32 or bf16
  const float* G;       // B*Opad*Ipad fp32
  void* Rout;           // B*Opad*Ipad, fp32 (FP32 path) or bf16
  float *L, *M, *V;     // K planes each, in blocks of kStateBlock coordinates (K = logits per coordinate)
  const uint8_t* J0;    // local shift: initial grid index of every coordinate (N bytes)
  float *S, *MS, *VS;   // one per scale group
  int* flag;            // sticky non-finite flag
  double* loss_part;    // backward: loss partial of (row, 256-column block), when want_loss
  int32_t want_loss;
  int64_t N;            // B*O*I
  int32_t rows;         // B*O
  int32_t O, I, Opad, Ipad, gs, w_bf16;
  uint64_t seed;
  float c[GSQ_MAX_LEVELS];    // the grid
  int32_t n_grid;
  // this step's sample(s)
  uint32_t t;
  int32_t noise;
  int32_t sample;             // forward: index of the independent draw
  int32_t samples;            // backward: number of draws averaged (G of draw m at G + m * g_stride)
  int64_t g_stride;
  float kappa, inv_tau;       // fp32 path of the BF16 precision
  double inv_tau_d;           // fp64 path of the FP32 precision
  // optimiser: Adam (step_* = lr / (1 - b1^n), rbc2 = 1/sqrt(1 - b2^n)) or Lion; decoupled decay
  int32_t lion;
  float lr, lr_s, b1, b2, eps, step_l, step_s, rbc2, wd;
  double step_l_d, step_s_d, rbc2_d;
  // sample of the next step, drawn by the backward kernel when fuse != 0
  int32_t fuse;
  uint32_t t_next;
  float kappa_n, inv_tau_n;
  double inv_tau_n_d;
};

struct Layer;
int64_t state_floats(const Layer& L);   // floats of one logit / moment array

struct Layer {
  gsq_config cfg;
  int64_t B, O, I, K, gs, Opad, Ipad, N, NG;   // K: logits per coordinate
  int n_grid;                                   // grid levels (code values)
  int relax;                                    // GSQ_RELAX_*
  bool bf16;        // precision == GSQ_PREC_BF16
  int w_bf16;
  void* W = nullptr;
  void* H = nullptr;
  float *L = nullptr, *M = nullptr, *V = nullptr;
  float *S = nullptr, *MS = nullptr, *VS = nullptr;
  void* R[2] = {nullptr, nullptr};
  float* G = nullptr;          // one padded gradient per sample slot
  double* partials = nullptr;  // loss partials of the contraction tiles (hard loss)
  double* loss_part = nullptr; // loss partials of the backward, one per row and 256 columns
  int64_t loss_cols = 0;       // 256-column blocks per row
  double* loss_stage = nullptr;    // chunk sums of the loss reduction
  unsigned* loss_tickets = nullptr;  // per layer: chunks summed so far (zero between launches)
  int sample_slots = 1;        // capacity of G in samples
  int last_sample = 0;         // slot holding the most recent step's last sample
  int64_t tiles_per_batch = 0;
  // contraction work split of a partly empty last round (see plan_contract_split)
  int split_full = 0, split_parts = 1;
  float* split_ws = nullptr;
  int* flag = nullptr;
  uint16_t* sb_d = nullptr;
  uint8_t* sb_sc = nullptr;
  uint8_t* codes = nullptr;
  uint8_t* J0 = nullptr;       // local shift: initial grid indices
  int64_t t = 0;
  int device = 0;         // HIP device the handle was created on
  int cur = 0;            // R buffer holding a prepared sample (when r_valid)
  bool r_valid = false;
  int64_t r_t = -1;
  float r_tau = 0.f, r_kappa = 0.f;
  int r_noise = 0;
  int last = -1;          // R buffer of the most recent step (-1: none)
  // kernel timing (gsq_timing)
  bool timing = false;
  std::vector<hipEvent_t> event_pool;
  std::vector<std::pair<int, std::pair<hipEvent_t, hipEvent_t>>> pending;
  double timed_ms[GSQ_NUM_KERNELS] = {0};
  int64_t timed_launches[GSQ_NUM_KERNELS] = {0};
};

// ---- launchers (gsq_elem.hip)
hipError_t launch_symmetrize_h(const float* Hin, void* Hout, int64_t B, int64_t I, int64_t Ipad,
                               bool bf16, hipStream_t s);
hipError_t launch_init_scales(const Layer& L, const float* scales_init, float cmax, hipStream_t s);
hipError_t launch_init_logits(const Layer& L, const double* mids, hipStream_t s);
hipError_t launch_forward(const Layer& L, const ElemArgs& a, hipStream_t s);
hipError_t launch_backward(const Layer& L, const ElemArgs& a, bool update_scales, hipStream_t s);
hipError_t launch_harden(const Layer& L, uint8_t* codes, void* Rh, hipStream_t s);
hipError_t launch_eff_scales(const Layer& L, float* out, hipStream_t s);
hipError_t launch_pack(const Layer& L, const uint8_t* codes, uint8_t* out, hipStream_t s);
hipError_t launch_state_io(const Layer& L, float* inter, float* planar, bool to_planar, hipStream_t s);
hipError_t launch_copy_residual(const Layer& L, const void* Rpad, void* out, hipStream_t s);
hipError_t launch_copy_grad(const Layer& L, const float* Gpad, float* out, hipStream_t s);
hipError_t launch_gumbel(const gsq_config& cfg, int64_t e0, int64_t count, int64_t t, float* out,
                         hipStream_t s);
ElemArgs base_args(const Layer& L);

// ---- launchers (gsq_contract.hip)
int64_t contract_tiles_per_batch(const Layer& L);
// Let the BF16 contraction use its 160 KB of LDS on the current device (called at init).
hipError_t prepare_contract_kernel();
int64_t loss_stage_size(const Layer& L);   // doubles
// Split the K range of the tiles of a last, at most half-full round of the GPU's num_cu
// compute units over 2 or 4 blocks each (BF16 precision, one layer, at least 128 K slabs per
// tile); sets split_full/_parts.
void plan_contract_split(Layer& L, int num_cu);
int64_t contract_split_ws_floats(const Layer& L);
hipError_t launch_contract(const Layer& L, const void* R, bool want_loss, int slot, hipStream_t s);
// Loss of each layer from the contraction's tile partials (slot 0) or, with from_rows, from the
// backward's row partials, times `scale`.
hipError_t launch_reduce_loss(const Layer& L, float* loss_out, bool from_rows, double scale,
                              hipStream_t s);
// The same with caller-chosen buffers: partials, chunk sums (>= the stage size of the reduction)
// and one ticket per layer (zero on entry, left at zero).
hipError_t launch_reduce_loss(const Layer& L, const double* part, double* stage, unsigned* tickets,
                              float* loss_out, bool from_rows, double scale, hipStream_t s);
int64_t loss_row_partials(const Layer& L);   // doubles written by the backward's loss terms
int64_t loss_row_stage(const Layer& L);      // chunk sums of their reduction

}  // namespace gsq
