// The dense contraction of the GSQ step: P = R H for every row of the residual R = W - W_hat,
// the gradient G = dL/dW_hat = -2 P (H symmetric) and, on request, per-tile partial sums of
// the loss tr(R H R^T) = sum(R * P) (Eq. 1 for a linear layer, H = X^T X).
//
// BF16 precision: R and H in bf16, products accumulated in fp32 on the matrix cores
// (v_mfma 32x32x16 bf16).  Because H is symmetric, column i of H is row i, so both operands
// are read along their contiguous dimension.
// FP32 precision: fp32 operands, fp64 accumulation on the vector units.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "gsq_device.hpp"
#include "gsq_internal.h"

namespace gsq {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = kTileM, BN = kTileN, BK = 64;
constexpr int A_STAGES = 3;                              // LDS ring of R's K slabs
constexpr int B_STAGES = 2;                              // LDS ring of H's K slabs
constexpr int ROW_BYTES = BK * 2;                        // one 64-wide bf16 row: a full cache line
constexpr int SLAB_BYTES = BM * ROW_BYTES;               // 32 KB per operand slab
constexpr int B_BASE = A_STAGES * SLAB_BYTES;            // H's ring after R's
constexpr size_t LDS_BYTES = (size_t)(A_STAGES + B_STAGES) * SLAB_BYTES;   // 160 KB
constexpr int LOADS_PER_OPERAND = SLAB_BYTES / 1024 / 4;   // 1 KB loads per wavefront per operand slab
constexpr int GROUP_M = 8;           // tile rows swept together for L2 reuse

// Sum over the workgroup into *out, through `red` (blockDim.x doubles of LDS, free to reuse).
__device__ __forceinline__ void block_sum_to(double x, double* out, double* red) {
  __syncthreads();
  red[threadIdx.x] = x;
  __syncthreads();
  for (int w = blockDim.x / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0];
}

// Position of block `bid` in the tile order.  Workgroups are handed to the 8 XCDs round-robin;
// renumbering so each XCD owns a contiguous range of the nblk blocks keeps the R and H panels a
// group of tiles shares in the same XCD's L2.
__device__ __forceinline__ int lin_of(int bid, int nblk) {
  return (nblk & 7) == 0 ? (bid & 7) * (nblk >> 3) + (bid >> 3) : bid;
}

// Tile at position `lin`: GROUP_M tile rows are swept together, column by column.
__device__ __forceinline__ void tile_at(int lin, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int per_group = GROUP_M * tiles_n;
  const int first_m = (lin / per_group) * GROUP_M;
  const int gsz = min(tiles_m - first_m, GROUP_M);
  const int r = lin % per_group;
  tm = first_m + r % gsz;
  tn = r / gsz;
}

// Work of one launch.  The first `full` blocks compute whole tiles (positions 0 .. full - 1).
// When the tiles do not fill a whole number of rounds of the GPU, the tiles of the last, partly
// empty round (positions full ..) are split along K: block full + q computes part q % split of
// tile full + q / split and writes its raw P to ws; k_contract_fixup adds the parts in order.
struct Split {
  int full;
  int split;    // 1: no split
  float* ws;    // (tiles - full) x split x 256 x 256 fp32
};

// Batches of layers (MoE experts): the tiles of each layer are grouped into blocks of bm x bn
// tiles (bm tile rows, bn tile columns, bm bn <= 32), one block per XCD at a time, so that the
// 32 CUs of an XCD work on one layer's 32 tiles together and its L2 holds bm R panels and bn H
// panels for them.  Block q goes to XCD q mod 8 (workgroup w runs on XCD w mod 8); the XCD's
// workgroups take its blocks in turn, 32 per block.
struct XcdBlocks {
  int on;
  int bm, bn;       // block shape in tiles
  int nbr, nbc;     // blocks per layer: rows, columns
  int nblocks;      // over all layers
};

// One 256 x 256 tile of G per workgroup; four wavefronts each own 128 x 128 as 4 x 4 MFMA
// 32x32x16 tiles.  K slabs 64 wide (whole 128-byte lines of R and H) move by direct global->LDS
// loads (16 bytes per lane, no staging registers) into a ring of three buffers for R and two for
// H, the whole 160 KB of LDS.  R's third buffer lets its slab k + 2 be loaded during the first
// half of slab k, H's during the second: the loads split evenly between the halves and R's get
// one and a half slabs of time to land.  The steady-state loop has no branches, so the fragment
// reads and slab loads are spread between the matrix-core instructions (scheduling groups)
// instead of stalling them.
//
// LDS layout of a slab: row r occupies 128 bytes as eight 16-byte chunks, chunk c stored at
// position c ^ f(r), f(r) = (r ^ (r >> 3)) & 7.  The fragment reads (consecutive rows, one
// chunk each) then fall on distinct banks for 8- and 16-lane access phases and for 32 or 64
// banks.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

// Global->LDS copy of one operand's slab rows 64 w .. 64 w + 63 (wave w): eight instructions of
// eight rows, 16 bytes per lane.  `src` is wave-uniform (the slab's first column); off[j] is the
// lane's element offset of instruction j, fixed for the whole K loop.
__device__ __forceinline__ void load_slab(const uint16_t* src, const uint32_t (&off)[8],
                                          uint8_t* lds_wave) {
#pragma unroll
  for (int j = 0; j < 8; ++j)
    __builtin_amdgcn_global_load_lds(src + off[j], lds_wave + j * 8 * ROW_BYTES, 16, 0, 0);
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

// Workgroup barrier for the slab ring: this wavefront's LDS reads are drained (its own
// global->LDS loads were waited for with wait_vm), then a plain s_barrier.  The signal fences
// keep the compiler from moving memory accesses across it; the waits are real instructions, so
// the compiler's own wait bookkeeping sees them.
__device__ __forceinline__ void slab_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt((15) | (7 << 4) | (0 << 8) | (3 << 14));   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// scheduling-group masks
constexpr int SG_MFMA = 0x008, SG_VMEM = 0x020, SG_DSR = 0x100;

// Epilogue of a tile: the raw P of a split tile's K part into the workspace, else G = -2 P and,
// on request, the tile's loss partial sum(R P).
// 32 x 32 accumulator layout: lane l, register r -> row 8*(r/4) + 4*(l/32) + r%4, column l%32.
__device__ __forceinline__ void finish_tile(f32x16 (&acc)[4][4], const uint16_t* R, float* G,
                                            double* partials, int64_t Opad, int64_t Ipad,
                                            int tiles_m, int tiles_n, int want_loss,
                                            const Split& sp, int64_t b, int tm, int tn, int part,
                                            int lin, int wm, int wn, int lane, uint8_t* smem) {
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  if (part >= 0) {   // raw P of this K part, tile-local row-major
    float* W_ = sp.ws + ((int64_t)(lin - sp.full) * sp.split + part) * (BM * BN);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          W_[(wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)) * BN + wn * 128 + j * 32 +
             (lane & 31)] = acc[i][j][r];
    return;
  }
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
  if (want_loss)
    block_sum_to(lsum, partials + b * (int64_t)tiles_m * tiles_n + tm * tiles_n + tn,
                 reinterpret_cast<double*>(smem));
}

// The tile of this workgroup: layer b, tile row tm, tile column tn, and for a split tile of the
// last round its K part (part >= 0) as slabs kb .. kb + nk - 1.  False: no tile (whole group).
__device__ __forceinline__ bool pick_tile(int tiles_m, int tiles_n, int64_t Ipad, const Split& sp,
                                          const XcdBlocks& xb, int64_t& b, int& tm, int& tn,
                                          int& part, int& kb, int& nk, int& lin) {
  b = blockIdx.z;
  nk = (int)(Ipad / BK);   // a multiple of 4 (Ipad is a multiple of 256)
  lin = 0;
  part = -1;
  kb = 0;
  if (xb.on) {
    const int x = blockIdx.x & 7, k = blockIdx.x >> 3;
    const int q = (k >> 5) * 8 + x, j = k & 31;
    if (q >= xb.nblocks || j >= xb.bm * xb.bn) return false;
    const int per_layer = xb.nbr * xb.nbc;
    b = q / per_layer;
    const int r = q - (int)b * per_layer;
    tm = (r / xb.nbc) * xb.bm + j % xb.bm;
    tn = (r % xb.nbc) * xb.bn + j / xb.bm;
    return tm < tiles_m && tn < tiles_n;
  }
  if ((int)blockIdx.x < sp.full) {
    lin = lin_of(blockIdx.x, sp.full);
  } else {   // a K part of a tile of the last round (XCD-contiguous numbering as well)
    const int nq = (int)gridDim.x - sp.full;
    const int q = lin_of(blockIdx.x - sp.full, nq);
    lin = sp.full + q / sp.split;
    part = q % sp.split;
    nk /= sp.split;
    kb = part * nk;
  }
  tile_at(lin, tiles_m, tiles_n, tm, tn);
  return true;
}

__global__ __launch_bounds__(256, 1) void k_contract_bf16(const uint16_t* __restrict__ R,
                                                          const uint16_t* __restrict__ H,
                                                          float* __restrict__ G,
                                                          double* __restrict__ partials,
                                                          int64_t Opad, int64_t Ipad, int tiles_m,
                                                          int tiles_n, int want_loss, Split sp,
                                                          XcdBlocks xb) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  int64_t b;
  int tm, tn, part, kb, nk, lin;
  if (!pick_tile(tiles_m, tiles_n, Ipad, sp, xb, b, tm, tn, part, kb, nk, lin)) return;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const uint16_t* A = R + b * Opad * Ipad + m0 * Ipad + (int64_t)kb * BK;
  const uint16_t* Bt = H + b * Ipad * Ipad + n0 * Ipad + (int64_t)kb * BK;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // lane offsets of the slab copies: row 64 wave + 8 j + lane / 8, swizzled 16-byte chunk
  uint32_t off[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = wave * 64 + j * 8 + (lane >> 3);
    // < 256 Ipad + 64 <= 2^32 for the widest layer the library accepts (I <= 2^24)
    off[j] = (uint32_t)row * (uint32_t)Ipad + (uint32_t)(((lane & 7) ^ swz(row)) * 8);
  }
#define GSQ_ISSUE_A(K) \
  load_slab(A + (int64_t)(K) * BK, off, smem + ((K) % A_STAGES) * SLAB_BYTES + wave * 64 * ROW_BYTES)
#define GSQ_ISSUE_B(K)                                                                   \
  load_slab(Bt + (int64_t)(K) * BK, off,                                                 \
            smem + B_BASE + ((K) % B_STAGES) * SLAB_BYTES + wave * 64 * ROW_BYTES)
  const int frow_a = wm * 128 + (lane & 31), frow_b = wn * 128 + (lane & 31);
  const int fchunk = lane >> 5;

// fragments of sub-steps 2 HALF and 2 HALF + 1 of slab K into register set S
#define GSQ_READ(S, K, HALF)                                                             \
  do {                                                                                   \
    const uint8_t* As_ = smem + ((K) % A_STAGES) * SLAB_BYTES;                           \
    const uint8_t* Bs_ = smem + B_BASE + ((K) % B_STAGES) * SLAB_BYTES;                  \
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
// interleave: 16 x (one MFMA, one LDS read), then 8 x (one MFMA, one global->LDS load) and 8
// MFMAs
#define GSQ_SCHED_LOADS_READS()                                                          \
  _Pragma("unroll") for (int i_ = 0; i_ < 16; ++i_) {                                    \
    __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);                                 \
    __builtin_amdgcn_sched_group_barrier(SG_DSR, 1, 0);                                  \
  }                                                                                      \
  _Pragma("unroll") for (int i_ = 0; i_ < 8; ++i_) {                                     \
    __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);                                 \
    __builtin_amdgcn_sched_group_barrier(SG_VMEM, 1, 0);                                 \
  }                                                                                      \
  __builtin_amdgcn_sched_group_barrier(SG_MFMA, 8, 0)

  // p: first half (sub-steps 0, 1) of the current slab; q: second half (sub-steps 2, 3)
  bf16x8 pa[2][4], pb[2][4], qa[2][4], qb[2][4];
  GSQ_ISSUE_A(0);
  GSQ_ISSUE_B(0);
  GSQ_ISSUE_A(1);
  GSQ_ISSUE_B(1);
  wait_vm<2 * LOADS_PER_OPERAND>();
  slab_barrier();
  GSQ_READ(p, 0, 0);
  // steady state: R's slab kt + 2 is loaded during the first half of slab kt (its buffer last
  // held slab kt - 1), H's during the second half (its buffer held slab kt, read by then)
  for (int kt = 0; kt < nk - 2; ++kt) {
    GSQ_READ(q, kt, 1);
    GSQ_ISSUE_A(kt + 2);
    GSQ_MFMA(p);
    GSQ_SCHED_LOADS_READS();
    __builtin_amdgcn_sched_barrier(0);   // every MFMA of this half is issued before the wait
    // slab kt+1 has landed (only R's slab kt+2 may be in flight), and every wavefront has read
    // slab kt
    wait_vm<LOADS_PER_OPERAND>();
    slab_barrier();
    GSQ_READ(p, kt + 1, 0);
    GSQ_ISSUE_B(kt + 2);
    GSQ_MFMA(q);
    GSQ_SCHED_LOADS_READS();
    __builtin_amdgcn_sched_barrier(0);
  }
  // the last two slabs: nothing more to load
  GSQ_READ(q, nk - 2, 1);
  GSQ_MFMA(p);
  wait_vm<0>();
  slab_barrier();
  GSQ_READ(p, nk - 1, 0);
  GSQ_MFMA(q);
  GSQ_READ(q, nk - 1, 1);
  GSQ_MFMA(p);
  GSQ_MFMA(q);
#undef GSQ_SCHED_LOADS_READS
#undef GSQ_MFMA
#undef GSQ_READ
#undef GSQ_ISSUE_A
#undef GSQ_ISSUE_B

  finish_tile(acc, R, G, partials, Opad, Ipad, tiles_m, tiles_n, want_loss, sp, b, tm, tn, part, lin,
              wm, wn, lane, smem);
}

// G = -2 (P_0 + ... + P_{split-1}) for the split tiles of the last round, parts added in order.
// Block (q, y) covers rows y * FIX_ROWS .. of split tile q, so the fixup spreads over enough
// workgroups to stream at the HBM rate.
constexpr int FIX_ROWS = 32;

__global__ __launch_bounds__(256) void k_contract_fixup(const float* __restrict__ ws,
                                                        float* __restrict__ G, int64_t Ipad,
                                                        int tiles_m, int tiles_n, Split sp) {
  const int q = blockIdx.x;
  int tm, tn;
  tile_at(sp.full + q, tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const float* src = ws + (int64_t)q * sp.split * (BM * BN);
  const int lo = blockIdx.y * FIX_ROWS * BN, hi = lo + FIX_ROWS * BN;
  for (int e = lo + threadIdx.x * 4; e < hi; e += 256 * 4) {
    float4 acc = *reinterpret_cast<const float4*>(src + e);
    for (int p = 1; p < sp.split; ++p) {
      const float4 v = *reinterpret_cast<const float4*>(src + (int64_t)p * (BM * BN) + e);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    const int lr = e / BN, lc = e % BN;
    *reinterpret_cast<float4*>(G + (m0 + lr) * Ipad + n0 + lc) =
        make_float4(-2.f * acc.x, -2.f * acc.y, -2.f * acc.z, -2.f * acc.w);
  }
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
  {
    __shared__ double red[256];
    block_sum_to(lsum, partials + (b * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x, red);
  }
}

// Loss of layer b = scale * the sum of its per_batch partials, in a fixed order, in one launch:
// block (c, b) sums chunk c (kChunk consecutive partials) into stage[b * nchunks + c]; the last
// block of layer b to finish (a ticket counter, reset by that block) sums the chunks in order.
constexpr int kPer = 8;                 // partials per thread, all loaded before summing
constexpr int kChunk = 256 * kPer;

__device__ __forceinline__ double block_tree_sum(double x) {
  __shared__ double red[256];
  red[threadIdx.x] = x;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__global__ void k_reduce_loss(const double* partials, int64_t per_batch, int nchunks,
                              double* stage, unsigned* tickets, double scale, float* loss_out,
                              int* flag) {
  const int64_t b = blockIdx.y, c = blockIdx.x;
  const int64_t lo = c * kChunk, hi = min(per_batch, lo + kChunk);
  double v[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int64_t i = lo + threadIdx.x + 256 * j;
    v[j] = i < hi ? partials[b * per_batch + i] : 0.0;
  }
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) s += v[j];
  const double tot = block_tree_sum(s);
  __shared__ unsigned ticket;
  if (threadIdx.x == 0) {
    stage[b * nchunks + c] = tot;
    __threadfence();                       // the chunk sum is visible before the ticket
    ticket = atomicAdd(&tickets[b], 1u);
  }
  __syncthreads();
  if (ticket != (unsigned)(nchunks - 1)) return;
  __threadfence();
  double t = 0.0;
  for (int i = threadIdx.x; i < nchunks; i += 256) t += __builtin_nontemporal_load(&stage[b * nchunks + i]);
  const double all = block_tree_sum(t);
  if (threadIdx.x == 0) {
    const float L = (float)(all * scale);
    loss_out[b] = L;
    if (!__builtin_isfinite(L)) *flag = 1;
    tickets[b] = 0u;
  }
}

}  // namespace

hipError_t prepare_contract_kernel() {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(k_contract_bf16),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)LDS_BYTES);
}

int64_t contract_tiles_per_batch(const Layer& L) {
  return L.bf16 ? (L.Opad / BM) * (L.Ipad / BN) : (L.Opad / TM) * (L.Ipad / TN);
}

hipError_t launch_contract(const Layer& L, const void* R, bool want_loss, int slot, hipStream_t s) {
  float* G = L.G + (int64_t)slot * L.B * L.Opad * L.Ipad;
  double* partials = L.partials;
  if (L.bf16) {
    const int tiles_m = (int)(L.Opad / BM), tiles_n = (int)(L.Ipad / BN);
    const int tiles = tiles_m * tiles_n;
    Split sp{tiles, 1, nullptr};
    if (L.split_parts > 1 && !want_loss) sp = Split{L.split_full, L.split_parts, L.split_ws};
    dim3 grid((unsigned)(sp.full + (tiles - sp.full) * sp.split), 1, (unsigned)L.B);
    XcdBlocks xb{0, 0, 0, 0, 0, 0};
    if (L.B > 1) {   // one layer's block of tiles per XCD at a time
      xb.on = 1;
      xb.bm = std::min(tiles_m, 8);
      xb.bn = std::min(tiles_n, 32 / xb.bm);
      xb.nbr = (tiles_m + xb.bm - 1) / xb.bm;
      xb.nbc = (tiles_n + xb.bn - 1) / xb.bn;
      xb.nblocks = (int)L.B * xb.nbr * xb.nbc;
      grid = dim3((unsigned)(8 * 32 * ((xb.nblocks + 7) / 8)), 1, 1);
    }
    hipLaunchKernelGGL(k_contract_bf16, grid, dim3(256), LDS_BYTES, s,
                       static_cast<const uint16_t*>(R), static_cast<const uint16_t*>(L.H), G,
                       partials, L.Opad, L.Ipad, tiles_m, tiles_n, want_loss ? 1 : 0, sp, xb);
    if (sp.split > 1) {
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(k_contract_fixup, dim3((unsigned)(tiles - sp.full), BM / FIX_ROWS), dim3(256), 0, s,
                         sp.ws, G, L.Ipad, tiles_m, tiles_n, sp);
    }
  } else {
    dim3 grid((unsigned)(L.Ipad / TN), (unsigned)(L.Opad / TM), (unsigned)L.B);
    hipLaunchKernelGGL(k_contract_f32, grid, dim3(256), 0, s, static_cast<const float*>(R),
                       static_cast<const float*>(L.H), G, partials, L.Opad, L.Ipad,
                       want_loss ? 1 : 0);
  }
  return hipGetLastError();
}

void plan_contract_split(Layer& L, int num_cu) {
  L.split_full = 0;
  L.split_parts = 1;
  if (!L.bf16 || L.B != 1 || num_cu <= 0) return;
  const int tiles = (int)((L.Opad / BM) * (L.Ipad / BN));
  const int rest = tiles % num_cu;
  if (tiles < num_cu || rest == 0 || rest > num_cu / 2) return;
  const int nk = (int)(L.Ipad / BK);
  if (nk < 128) return;   // short K loops: the partial-product traffic would cost more than it saves
  int split = 1;
  for (int s = 2; s <= 4; s *= 2)
    if (rest * s <= num_cu && nk % s == 0 && nk / s >= 2) split = s;
  if (split == 1) return;
  L.split_full = tiles - rest;
  L.split_parts = split;
}

int64_t contract_split_ws_floats(const Layer& L) {
  if (L.split_parts <= 1) return 0;
  const int tiles = (int)((L.Opad / BM) * (L.Ipad / BN));
  return (int64_t)(tiles - L.split_full) * L.split_parts * BM * BN;
}

int64_t loss_stage_size(const Layer& L) {
  const int64_t most = std::max<int64_t>(L.O * L.loss_cols, contract_tiles_per_batch(L));
  return L.B * ((most + kChunk - 1) / kChunk);
}

int64_t loss_row_partials(const Layer& L) { return L.B * L.O * L.loss_cols; }

int64_t loss_row_stage(const Layer& L) {
  return L.B * ((L.O * L.loss_cols + kChunk - 1) / kChunk);
}

hipError_t launch_reduce_loss(const Layer& L, float* loss_out, bool from_rows, double scale,
                              hipStream_t s) {
  return launch_reduce_loss(L, from_rows ? L.loss_part : L.partials, L.loss_stage, L.loss_tickets,
                            loss_out, from_rows, scale, s);
}

hipError_t launch_reduce_loss(const Layer& L, const double* part, double* stage, unsigned* tickets,
                              float* loss_out, bool from_rows, double scale, hipStream_t s) {
  const int64_t per_batch = from_rows ? L.O * L.loss_cols : contract_tiles_per_batch(L);
  const int nchunks = (int)((per_batch + kChunk - 1) / kChunk);
  hipLaunchKernelGGL(k_reduce_loss, dim3((unsigned)nchunks, (unsigned)L.B), dim3(256), 0, s, part,
                     per_batch, nchunks, stage, tickets, scale, loss_out, L.flag);
  return hipGetLastError();
}

}  // namespace gsq
