// The dense contraction of the GSQ step: P = R H for every row of the residual R = W - W_hat,
// the gradient G = dL/dW_hat = -2 P (H symmetric) and, on request, per-tile partial sums of
// the loss tr(R H R^T) = sum(R * P) (Eq. 1 for a linear layer, H = X^T X).
//
// BF16 precision: R and H in bf16, products accumulated in fp32 on the matrix cores
// (v_mfma 32x32x16 bf16).  Because H is symmetric, column i of H is row i, so both operands
// are read along their contiguous dimension.
// FP32 precision: fp32 operands, fp64 accumulation on the vector units.
#include <hip/hip_runtime.h>

#include "gsq_device.hpp"
#include "gsq_internal.h"

namespace gsq {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = kTileM, BN = kTileN, BK = 64;
constexpr int STAGES = 2;                                // LDS ring of K slabs
constexpr int ROW_BYTES = BK * 2;                        // one 64-wide bf16 row: a full cache line
constexpr int SLAB_BYTES = BM * ROW_BYTES;               // 32 KB per operand per stage
constexpr size_t LDS_BYTES = (size_t)STAGES * 2 * SLAB_BYTES;
constexpr int LOADS_PER_STAGE = 2 * SLAB_BYTES / 1024 / 4;   // 1 KB loads per wavefront per stage
constexpr int GROUP_M = 8;           // tile rows swept together for L2 reuse

__device__ __forceinline__ void block_sum_to(double x, double* out) {
  __shared__ double red[256];
  red[threadIdx.x] = x;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0];
}

// Tile of block `bid`.  Workgroups are handed to the 8 XCDs round-robin; renumbering so
// each XCD owns a contiguous range, then sweeping GROUP_M tile rows at a time, keeps the
// R and H panels a group shares in the same XCD's L2.
__device__ __forceinline__ void tile_of(int bid, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nblk = tiles_m * tiles_n;
  int lin = bid;
  if ((nblk & 7) == 0) lin = (bid & 7) * (nblk >> 3) + (bid >> 3);
  const int per_group = GROUP_M * tiles_n;
  const int first_m = (lin / per_group) * GROUP_M;
  const int gsz = min(tiles_m - first_m, GROUP_M);
  const int r = lin % per_group;
  tm = first_m + r % gsz;
  tn = r / gsz;
}

// One 256 x 256 tile of G per workgroup; four wavefronts each own 128 x 128 as 4 x 4 MFMA
// 32x32x16 tiles.  K slabs 64 wide (whole 128-byte lines of R and H) stream through two LDS
// buffers by direct global->LDS loads (16 bytes per lane, no staging registers).
//
// LDS layout of a slab: row r occupies 128 bytes as eight 16-byte chunks, chunk c stored at
// position c ^ f(r), f(r) = (r ^ (r >> 3)) & 7.  The fragment reads (consecutive rows, one
// chunk each) then fall on distinct banks for 8- and 16-lane access phases and for 32 or 64
// banks.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

__device__ __forceinline__ void load_slab(const uint16_t* src, int64_t ld, int64_t k0,
                                          uint8_t* lds, int wave, int lane) {
  // wave w fills rows 64 w .. 64 w + 63, eight rows (1 KB of LDS) per instruction
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = wave * 64 + j * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ swz(row);
    const uint16_t* g = src + row * ld + k0 + chunk * 8;
    __builtin_amdgcn_global_load_lds(g, lds + (wave * 64 + j * 8) * ROW_BYTES, 16, 0, 0);
  }
}

__device__ __forceinline__ bf16x8 read_frag(const uint8_t* lds, int row, int chunk) {
  return *reinterpret_cast<const bf16x8*>(lds + row * ROW_BYTES + ((chunk ^ swz(row)) << 4));
}

// Wait until at most n of this wavefront's vector-memory loads are outstanding (loads complete
// in issue order), leaving LDS and scalar counters alone.
template <int n>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
}

// Workgroup barrier for the slab ring.  The wavefront's own global->LDS loads have been
// waited for (wait_vm) and its LDS reads are drained here; a plain s_barrier then suffices.
// (__syncthreads would also drain every in-flight slab of the ring.)  The memory clobber
// keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void slab_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__global__ __launch_bounds__(256, 1) void k_contract_bf16(const uint16_t* __restrict__ R,
                                                          const uint16_t* __restrict__ H,
                                                          float* __restrict__ G,
                                                          double* __restrict__ partials,
                                                          int64_t Opad, int64_t Ipad, int tiles_m,
                                                          int tiles_n, int want_loss) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int64_t b = blockIdx.z;
  int tm, tn;
  tile_of(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const uint16_t* A = R + b * Opad * Ipad + m0 * Ipad;
  const uint16_t* Bt = H + b * Ipad * Ipad + n0 * Ipad;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int64_t nk = Ipad / BK;   // a multiple of 4 (Ipad is a multiple of 256)
  auto issue = [&](int64_t k) {
    uint8_t* st = smem + (k % STAGES) * 2 * SLAB_BYTES;
    load_slab(A, Ipad, k * BK, st, wave, lane);
    load_slab(Bt, Ipad, k * BK, st + SLAB_BYTES, wave, lane);
  };
  const int frow_a = wm * 128 + (lane & 31), frow_b = wn * 128 + (lane & 31);
  const int fchunk = lane >> 5;

// fragments of sub-steps 2 HALF and 2 HALF + 1 of slab K into register set S
#define GSQ_READ(S, K, HALF)                                                             \
  do {                                                                                   \
    const uint8_t* As_ = smem + ((K) % STAGES) * 2 * SLAB_BYTES;                         \
    const uint8_t* Bs_ = As_ + SLAB_BYTES;                                               \
    _Pragma("unroll") for (int h = 0; h < 2; ++h)                                        \
      _Pragma("unroll") for (int i = 0; i < 4; ++i) {                                    \
        const int c_ = (2 * (HALF) + h) * 2 + fchunk;                                    \
        S##a[h][i] = read_frag(As_, frow_a + i * 32, c_);                                \
        S##b[h][i] = read_frag(Bs_, frow_b + i * 32, c_);                                \
      }                                                                                  \
  } while (0)
#define GSQ_MFMA(S)                                                                      \
  _Pragma("unroll") for (int h = 0; h < 2; ++h)                                          \
    _Pragma("unroll") for (int i = 0; i < 4; ++i)                                        \
      _Pragma("unroll") for (int j = 0; j < 4; ++j)                                      \
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(S##a[h][i], S##b[h][j], acc[i][j], 0, 0, 0)

  // p: first half (sub-steps 0, 1) of the current slab; q: second half (sub-steps 2, 3)
  bf16x8 pa[2][4], pb[2][4], qa[2][4], qb[2][4];
  issue(0);
  issue(1);
  wait_vm<LOADS_PER_STAGE>();
  slab_barrier();
  GSQ_READ(p, 0, 0);
  for (int64_t kt = 0; kt < nk; ++kt) {
    // phase 1: read the second half of slab kt while its first half feeds the matrix cores
    GSQ_READ(q, kt, 1);
    GSQ_MFMA(p);
    // phase 2: slab kt+1 (issued one slab ago) must have landed, and every wavefront's reads
    // of slab kt must have returned before its buffer is refilled with slab kt+2
    if (kt + 1 < nk) {
      wait_vm<0>();
      slab_barrier();
      if (kt + 2 < nk) issue(kt + 2);
      GSQ_READ(p, kt + 1, 0);
    }
    GSQ_MFMA(q);
  }
#undef GSQ_MFMA
#undef GSQ_READ

  // 32 x 32 accumulator layout: lane l, register r -> row 8*(r/4) + 4*(l/32) + r%4, column l%32
  float* Gb = G + b * Opad * Ipad;
  const uint16_t* Rb = R + b * Opad * Ipad;
  double lsum = 0.0;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int64_t col = n0 + wn * 128 + j * 32 + (lane & 31);
        const float p = acc[i][j][r];
        Gb[row * Ipad + col] = -2.f * p;
        if (want_loss) lsum += (double)bf16_to_f32(Rb[row * Ipad + col]) * (double)p;
      }
  if (want_loss) block_sum_to(lsum, partials + b * (int64_t)tiles_m * tiles_n + tm * tiles_n + tn);
}

// FP32 precision: 64 x 64 tile per workgroup, 4 x 4 outputs per thread, fp64 accumulation.
constexpr int TM = 64, TN = 64, TK = 16;

__global__ __launch_bounds__(256) void k_contract_f32(const float* __restrict__ R,
                                                      const float* __restrict__ H,
                                                      float* __restrict__ G,
                                                      double* __restrict__ partials, int64_t Opad,
                                                      int64_t Ipad, int want_loss) {
  __shared__ float As[TK][TM + 1];
  __shared__ float Bs[TK][TN + 1];
  const int64_t b = blockIdx.z;
  const int64_t m0 = (int64_t)blockIdx.y * TM, n0 = (int64_t)blockIdx.x * TN;
  const float* A = R + b * Opad * Ipad + m0 * Ipad;
  const float* Bt = H + b * Ipad * Ipad + n0 * Ipad;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  double acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int64_t k0 = 0; k0 < Ipad; k0 += TK) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i, row = c >> 4, k = c & 15;
      As[k][row] = A[row * Ipad + k0 + k];
      Bs[k][row] = Bt[row * Ipad + k0 + k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; ++k) {
      double av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { av[i] = As[k][ty * 4 + i]; bv[i] = Bs[k][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fma(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
  double lsum = 0.0;
  float* Gb = G + b * Opad * Ipad;
  const float* Rb = R + b * Opad * Ipad;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
      Gb[row * Ipad + col] = (float)(-2.0 * acc[i][j]);
      if (want_loss) lsum += (double)Rb[row * Ipad + col] * acc[i][j];
    }
  if (want_loss)
    block_sum_to(lsum, partials + (b * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x);
}

// Loss of layer b = mean over the samples of the sum of its tile partials, in a fixed order.
// Partials of sample m, layer b start at (m * B + b) * per_batch.
__global__ void k_reduce_loss(const double* partials, int64_t per_batch, int64_t B, int samples,
                              float* loss_out, int* flag) {
  const int64_t b = blockIdx.x;
  double s = 0.0;
  for (int m = 0; m < samples; ++m)
    for (int64_t i = threadIdx.x; i < per_batch; i += 256) s += partials[(m * B + b) * per_batch + i];
  __shared__ double red[256];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const float L = (float)(red[0] / samples);
    loss_out[b] = L;
    if (!__builtin_isfinite(L)) *flag = 1;
  }
}

}  // namespace

int64_t contract_tiles_per_batch(const Layer& L) {
  return L.bf16 ? (L.Opad / BM) * (L.Ipad / BN) : (L.Opad / TM) * (L.Ipad / TN);
}

hipError_t launch_contract(const Layer& L, const void* R, bool want_loss, int slot, hipStream_t s) {
  float* G = L.G + (int64_t)slot * L.B * L.Opad * L.Ipad;
  double* partials = L.partials + (int64_t)slot * L.B * L.tiles_per_batch;
  if (L.bf16) {
    static bool attr_set = false;
    if (!attr_set) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(k_contract_bf16),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)LDS_BYTES);
      if (e != hipSuccess) return e;
      attr_set = true;
    }
    const int tiles_m = (int)(L.Opad / BM), tiles_n = (int)(L.Ipad / BN);
    dim3 grid((unsigned)(tiles_m * tiles_n), 1, (unsigned)L.B);
    hipLaunchKernelGGL(k_contract_bf16, grid, dim3(256), LDS_BYTES, s,
                       static_cast<const uint16_t*>(R), static_cast<const uint16_t*>(L.H), G,
                       partials, L.Opad, L.Ipad, tiles_m, tiles_n, want_loss ? 1 : 0);
  } else {
    dim3 grid((unsigned)(L.Ipad / TN), (unsigned)(L.Opad / TM), (unsigned)L.B);
    hipLaunchKernelGGL(k_contract_f32, grid, dim3(256), 0, s, static_cast<const float*>(R),
                       static_cast<const float*>(L.H), G, partials, L.Opad, L.Ipad,
                       want_loss ? 1 : 0);
  }
  return hipGetLastError();
}

hipError_t launch_reduce_loss(const Layer& L, float* loss_out, int samples, hipStream_t s) {
  hipLaunchKernelGGL(k_reduce_loss, dim3((unsigned)L.B), dim3(256), 0, s, L.partials,
                     contract_tiles_per_batch(L), L.B, samples, loss_out, L.flag);
  return hipGetLastError();
}

}  // namespace gsq
