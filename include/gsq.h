/*
 * gsq.h -- C ABI of the GSQ layer-step library for MI355X (gfx950).
 *
 * The library optimises one linear layer (or a batch of independent layers,
 * e.g. the routed experts of an MoE block) with Gumbel-Softmax Quantization
 * (arXiv 2604.18556): find per-group scales s and per-coordinate grid codes q
 * minimising the layer-output error of Eq. 1 on calibration data, under the
 * b-bit scalar constraint W_hat = s * c[q] of Eq. 5 (§3.2), with groups of
 * consecutive weights along each row (§4.1).  For a linear layer with
 * calibration inputs X the objective of Eq. 1 is tr((W - W_hat) H (W - W_hat)^T)
 * with H = X^T X, which is what the caller supplies.
 *
 * Every call only enqueues work on the caller's HIP stream and returns; the
 * outputs are valid once the stream reaches that point.  Calls that must read
 * a device result first (gsq_check, gsq_harden, gsq_pack, gsq_get_state)
 * synchronise the stream themselves and say so.  Functions never throw and
 * never abort; each returns a gsq_status and, on error, leaves a message for
 * gsq_last_error() (thread-local).  Validation errors are returned before
 * anything is enqueued or allocated.
 *
 * Pointers named "device" must point to device memory of the current HIP
 * device (hipMalloc, torch CUDA tensors); "host" pointers to host memory.
 * A handle must not be used from two threads at once; separate handles are
 * independent.  All row-major arrays are dense (no strides).
 */
#ifndef GSQ_H
#define GSQ_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gsq_layer gsq_layer; /* opaque; owns every internal device buffer */

typedef enum {
  GSQ_OK = 0,
  GSQ_EINVAL = -1,        /* invalid argument or configuration                         */
  GSQ_ENOMEM = -2,        /* a device allocation failed                                */
  GSQ_EHIP = -3,          /* a HIP runtime call failed; gsq_last_error() has its text  */
  GSQ_ENONFINITE = -4,    /* a loss, gradient, updated parameter or fp16 scale was
                             not finite (sticky until the handle is destroyed)         */
  GSQ_EUNSUPPORTED = -5   /* valid request the library does not implement              */
} gsq_status;

enum { GSQ_LAYOUT_GROUP = 0, GSQ_LAYOUT_SUPERBLOCK = 1, GSQ_LAYOUT_BASE3 = 2 };
enum { GSQ_PREC_FP32 = 0, GSQ_PREC_BF16 = 1 };
enum { GSQ_DT_FP32 = 0, GSQ_DT_BF16 = 1 };
enum { GSQ_OPT_ADAM = 0, GSQ_OPT_LION = 1 };

/* How a coordinate's choice of grid level is relaxed.
 * GRID:    one categorical over all n_levels levels (Alg. 1 over the grid of Eq. 5, §3.2);
 *          n_levels logits per coordinate, 2 <= n_levels <= 8.
 * SHIFT:   the local-shift relaxation of §3.2 (Eq. 6) for wider grids: 5 logits per
 *          coordinate over the index shifts delta = -2..2 around a fixed initial index j0
 *          (the round-to-nearest code); logit k stands for the level
 *          c[clip(j0 + delta_k, 0, n_levels - 1)].  2 <= n_levels <= 16.
 * TERNARY: the mask x sign form of §3.1 (Eq. 2, Alg. 2): two logits per coordinate, l_m and
 *          l_b, each relaxed as a two-value Gumbel-Softmax with logits {-l, l}; the soft
 *          weight is s m~ b~ with m~ over {0, 1} and b~ over {-1, 1}.  Levels must be exactly
 *          {-1, 0, 1}; codes index them. */
enum { GSQ_RELAX_GRID = 0, GSQ_RELAX_SHIFT = 1, GSQ_RELAX_TERNARY = 2 };
#define GSQ_MAX_LEVELS 16
#define GSQ_SHIFT_WINDOW 5

/* Layer configuration (read at gsq_layer_init; copied). */
typedef struct {
  int32_t  batch;          /* independent layers sharing the configuration (>= 1)           */
  int32_t  out_features;   /* O (>= 1)                                                      */
  int32_t  in_features;    /* I; multiple of group_size (GROUP) or of 256 (SUPERBLOCK)      */
  int32_t  n_levels;       /* n: grid cardinality |G_b| of Eq. 5 (limits per relaxation)    */
  float    levels[GSQ_MAX_LEVELS]; /* c_0 < ... < c_{n-1}, finite, not all zero              */
  int32_t  group_size;     /* GROUP, BASE3: 16, 32, 64, 128 or 256 consecutive inputs per
                              scale; SUPERBLOCK: ignored (16-weight sub-blocks)             */
  int32_t  layout;         /* GSQ_LAYOUT_*: GROUP = b-bit codes and one fp16 scale per group
                              (Tab. 1 format); SUPERBLOCK = 256-weight records of 16
                              sub-blocks, each with a 6-bit scale times one fp16 scale per
                              record (K-quant style, §4.4; n_levels <= 8); BASE3 = as GROUP
                              but five 3-level codes per byte (n_levels == 3, 1.6 bits)     */
  int32_t  precision;      /* GSQ_PREC_*: type of the residual R and of H in the contraction.
                              BF16: bf16 operands, fp32 accumulation on the matrix cores,
                              fp32 elementwise arithmetic with hardware log/exp.
                              FP32: fp32 operands, fp64 accumulation, fp64 elementwise.     */
  uint64_t seed;           /* key of the Philox4x32-10 noise generator                      */
  float    alpha;          /* warm-start strength of Eq. 4 (the paper uses 6 for 2/3-bit)   */
  float    sigma_init;     /* overall logit scale of Eq. 4                                  */
  int32_t  init_noise;     /* 1: add N(0,1) noise to the initial logits (Eq. 4); 0: none    */
  int32_t  relaxation;     /* GSQ_RELAX_*; the initial logits follow the warm start of each:
                              GRID: App. A's Gaussian prior -(c_k - c_q0)^2/2 around the
                              round-to-nearest code q0; SHIFT: the prior -delta^2/2 centred at
                              delta = 0 (App. A, b > 2), j0 = q0; TERNARY: Eq. 3's +-1 / 0
                              mask and sign logits of q0.  Then l = sigma_init (eps + alpha
                              prior) (Eq. 4; GRID and SHIFT priors are mean-subtracted).    */
} gsq_config;

/* Scalars of one optimisation step (host values; the schedule lives with the caller). */
typedef struct {
  float   tau;             /* temperature of Alg. 1 (> 0)                                   */
  float   kappa;           /* logit ("noise") scale of Alg. 1 (finite)                      */
  float   lr_logits;       /* Adam step size of the logits (>= 0)                           */
  float   lr_scales;       /* Adam step size of the scales; 0 freezes them (required for
                              SUPERBLOCK, whose scales stay in their 6-bit grid)            */
  float   beta1, beta2;    /* Adam moment decays, in [0, 1)                                 */
  float   eps;             /* Adam denominator constant (> 0)                               */
  int32_t gumbel_noise;    /* 1: sample the noise of Alg. 1 (GRID, SHIFT: g ~ Gumbel(0,1)
                              per logit; TERNARY: one Logistic(0,1) value per binary pair,
                              as gsq_gumbel describes); 0: no noise                         */
  float   tau_next;        /* temperature of the NEXT call's step, or 0 if unknown.  When
                              the next call passes exactly (tau_next, kappa_next) the sample
                              of that step has already been drawn by this one, saving one
                              pass over the logits.  Results are identical either way.      */
  float   kappa_next;      /* logit scale of the next step (used when tau_next > 0)         */
  int32_t optimizer;       /* GSQ_OPT_ADAM: Adam, bias-corrected (AdamW when weight_decay > 0,
                              the paper's ablation, App. B); GSQ_OPT_LION: Lion, the paper's
                              optimiser (§3.3): theta -= lr (sign(beta1 m + (1-beta1) g)
                              + weight_decay theta), then m = beta2 m + (1-beta2) g; eps and
                              the second moment are unused                                   */
  float   weight_decay;    /* decoupled weight decay on logits and scales (>= 0)            */
  int32_t samples;         /* M independent noise draws this step, 0 or 1 = one draw, at most
                              GSQ_MAX_SAMPLES: gradients and the reported loss are averaged
                              over the M samples (§3.3, gradient accumulation with resampled
                              noise).  Each extra sample costs one more forward pass and one
                              more contraction; buffers for M samples are allocated on the
                              first step that asks for them.                                  */
} gsq_step_params;

#define GSQ_MAX_SAMPLES 16

/*
 * Create a layer.  W: device, batch x O x I row-major, fp32 or bf16 (w_dtype).
 * H: device fp32, batch x I x I row-major; only its symmetric part (H + H^T)/2
 * matters and the library keeps that (in the precision's type).
 * scales_init: device fp32 batch x O x (I/group_size), or NULL for
 * round-to-nearest absmax scales s = max|W_group| / max_k |c_k| (1 for an all-zero
 * group); must be NULL for SUPERBLOCK.  The logits start from the Gaussian prior
 * around the round-to-nearest codes (App. A) plus Eq. 4's noise; moments are zero,
 * the step counter t is 0.  W and H are copied: the caller may free them once the
 * stream has passed this call.  On success *out receives the handle.
 */
gsq_status gsq_layer_init(const gsq_config* cfg, const void* W, int32_t w_dtype, const float* H,
                          const float* scales_init, hipStream_t stream, gsq_layer** out);

/*
 * One optimisation step (Alg. 1 sample, Eq. 1 loss, gradient, optimiser; the loop body of
 * Alg. 2, generalised to n levels by §3.2): draws g for step t, forms the soft weight
 * (GRID, SHIFT: s * sum_k p_k c_k over the coordinate's candidate levels; TERNARY:
 * s m~ b~), the residual R, P = R H, the loss tr(R H R^T), the gradients of the logits
 * and scales, applies the optimiser (bias correction at step t+1) and advances t.
 * loss_out: device fp32[batch] receiving the loss of this step's sample(s) before the
 * update, or NULL to skip computing it.
 */
gsq_status gsq_step(gsq_layer* h, const gsq_step_params* p, float* loss_out, hipStream_t stream);

/*
 * gsq_step for callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  The same step, with the same results bit for
 * bit, but it allocates nothing: the scratch of the loss reduction (row partials, chunk sums, one
 * ticket per layer) lives in a static device array of the library, about 33 MiB per GPU, held
 * until the process ends, instead of in the handle's buffers; and the per-sample gradient
 * buffers are never grown.
 * Limits (GSQ_EINVAL before anything is enqueued): samples at most the most any earlier gsq_step
 * on this handle used (1 for a new handle); with loss_out, batch * O * ceil(I / 256) <= 4194304
 * row partials, batch * ceil(O * ceil(I / 256) / 2048) <= 65536 chunk sums and batch <= 65536.
 * The handle's device must be current.  Every call on one GPU shares that GPU's scratch, which
 * keeps the last call's contents: calls that overlap on one GPU (other streams, threads or
 * handles) race, and the caller must order them.
 */
gsq_status gsq_step_static(gsq_layer* h, const gsq_step_params* p, float* loss_out,
                           hipStream_t stream);

/*
 * Harden (the final step of Alg. 2): codes into `codes` (device u8, batch x O x I, or NULL),
 * code = grid level index.  GRID: argmax_k logits (ties to the lowest k); SHIFT:
 * clip(j0 + delta*) with delta* the argmax shift (ties to the lowest); TERNARY: mask
 * l_m >= 0 and sign + if l_b >= 0 else -, code 1 + mask * sign.  Effective scales
 * into `scales` (device fp32, batch x O x (I/group_size) -- GROUP: the fp16-rounded
 * scales, SUPERBLOCK: d * sc per 16-weight sub-block; or NULL); the hard loss
 * tr(R H R^T) with R = W - s c[q] into hard_loss_out (device fp32[batch], or NULL).
 * Synchronises the stream; returns GSQ_ENONFINITE if a scale overflows fp16 or the
 * sticky non-finite flag is set.
 */
gsq_status gsq_harden(gsq_layer* h, uint8_t* codes, float* scales, float* hard_loss_out,
                      hipStream_t stream);

/* Bytes gsq_pack writes for this configuration (0 if the configuration is invalid).
 * GROUP: batch*O*I*b/8 code bytes (b = ceil(log2 n_levels)) + 2*batch*O*(I/group_size) scale
 * bytes; BASE3: ceil(batch*O*I/5) code bytes + the same scale bytes; SUPERBLOCK: 110 bytes per
 * 256 weights. */
size_t gsq_packed_size(const gsq_config* cfg);

/*
 * Pack the hardened layer into `packed` (device, >= gsq_packed_size bytes, any alignment):
 * the deployment formats of the quantized weights -- Tab. 1's b-bit codes plus one 16-bit
 * scale per group (b + 16/gs bits per parameter, ternary at 1.6 + 16/gs), and the
 * K-quant-style super-blocks of §4.4 and App. E, into which the optimised codes are projected
 * back.  GROUP: one little-endian bitstream of b-bit codes (code = level index) over all
 * coordinates in row-major order, then the fp16 scales row-major.  BASE3: the codes
 * t in {0, 1, 2} in row-major order, five per byte, byte n = sum_j t_{5n+j} 3^j (the last
 * byte padded with zero codes), then the fp16 scales row-major.  SUPERBLOCK: per
 * 256 consecutive weights of a row, [fp16 d][16 x 6-bit sc, LSB first][256 x 3-bit
 * codes, LSB first] = 110 bytes, records row-major.  Synchronises the stream.
 */
gsq_status gsq_pack(gsq_layer* h, void* packed, size_t packed_bytes, hipStream_t stream);

/*
 * Copy the optimiser state out (device pointers, any may be NULL):
 * logits, m, v: fp32 batch x O x I x K with K the logits per coordinate (GRID: n_levels,
 * SHIFT: 5, TERNARY: 2 as (l_m, l_b)); scales, m_s, v_s: fp32 batch x O x (I/gs)
 * (gs = 16 for SUPERBLOCK); base: SHIFT only, u8 batch x O x I, the initial grid index j0
 * of every coordinate (must be NULL otherwise); t: host int64.  Synchronises the stream.
 */
gsq_status gsq_get_state(gsq_layer* h, float* logits, float* m, float* v, float* scales,
                         float* m_s, float* v_s, uint8_t* base, int64_t* t, hipStream_t stream);

/* Overwrite the state (same layouts; NULL leaves that part unchanged; t >= 0).  Every base
 * index should be < n_levels: the kernels read a larger one as n_levels - 1.  Invalid
 * arguments return before anything is enqueued. */
gsq_status gsq_set_state(gsq_layer* h, const float* logits, const float* m, const float* v,
                         const float* scales, const float* m_s, const float* v_s,
                         const uint8_t* base, int64_t t, hipStream_t stream);

/*
 * Intermediates of the most recent gsq_step (device pointers, either may be NULL):
 * residual R = W - W_hat of that step's (last) sample, batch x O x I, in the precision's
 * type (fp32 or bf16); grad = dL/dW_hat = -2 R H of the same sample, fp32 batch x O x I.
 * GSQ_EINVAL if no step has run since init / set_state / harden.
 */
gsq_status gsq_get_intermediates(gsq_layer* h, void* residual, float* grad, hipStream_t stream);

/*
 * The noise the step kernels draw (Alg. 1): for the `count` coordinates starting at global
 * index e0 (e = ((b*O)+o)*I + i) at step t, Z values each, into g_out (device fp32,
 * count x Z).  GRID, SHIFT: Z = the logits per coordinate (n_levels, 5) Gumbel(0,1) values
 * g = -ln(-ln u).  TERNARY: Z = 2 Logistic(0,1) values d = ln u - ln(1 - u), the mask pair's
 * then the sign pair's: a two-value relaxation with logits {-l, l} is a sigmoid of
 * 2 kappa l + g1 - g0 (§3), so each pair draws the difference of its two Gumbel values, which
 * has this law, as one value.  Uses cfg's seed and precision (FP32: evaluated in fp64 and
 * rounded once; BF16: hardware log2).
 */
gsq_status gsq_gumbel(const gsq_config* cfg, int64_t e0, int64_t count, int64_t t, float* g_out,
                      hipStream_t stream);

/* Kernels the library launches, as counted by gsq_timing_read. */
enum {
  GSQ_KERNEL_INIT = 0,      /* H symmetrisation, scale and logit initialisation        */
  GSQ_KERNEL_FORWARD = 1,   /* the sample of Alg. 1 and the residual R                 */
  GSQ_KERNEL_CONTRACT = 2,  /* P = R H, G = -2 P (hard loss: + loss partials)           */
  GSQ_KERNEL_REDUCE = 3,    /* loss partials -> loss                                    */
  GSQ_KERNEL_BACKWARD = 4,  /* gradient + optimiser + loss terms (+ the next sample)    */
  GSQ_KERNEL_HARDEN = 5,    /* codes, effective scales, hard residual                   */
  GSQ_KERNEL_PACK = 6,      /* bitstream / base-3 / super-block packing                 */
  GSQ_NUM_KERNELS = 7
};

/*
 * Kernel timing.  gsq_timing(h, 1) makes every later call record a HIP event pair
 * around each kernel it enqueues (on the caller's stream); gsq_timing(h, 0) stops.
 * gsq_timing_read synchronises `stream`, adds the elapsed time (ms) and the launch
 * count of each kernel kind since the last reset into ms[GSQ_NUM_KERNELS] and
 * launches[GSQ_NUM_KERNELS] (host arrays, either may be NULL), and clears them if
 * reset != 0.
 */
gsq_status gsq_timing(gsq_layer* h, int32_t enable);
gsq_status gsq_timing_read(gsq_layer* h, double* ms, int64_t* launches, int32_t reset,
                           hipStream_t stream);

/* Synchronise the stream and report the sticky non-finite flag (GSQ_OK or GSQ_ENONFINITE). */
gsq_status gsq_check(gsq_layer* h, hipStream_t stream);

/* Free every buffer of the handle (NULL-safe; synchronises the device). */
gsq_status gsq_layer_destroy(gsq_layer* h);

/* Message of the last error on this thread ("" if none). */
const char* gsq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GSQ_H */
