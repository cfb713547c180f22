// gemm_producer.h - the producer: a bf16 MFMA GEMM for gfx950 whose
// workgroups take their output blocks in a chosen traversal order and
// publish a ready flag per 128 x 128 tile (paper Sections 3.1 and 4.2).
//
// One workgroup computes a BM x BN block of C = A B (A: M x K, B: K x N, both
// row-major bf16) with 4 waves in a 2 x 2 arrangement; each wave owns a
// (BM/2) x (BN/2) sub-block as 32 x 32 MFMA accumulators
// (v_mfma_f32_32x32x16_bf16, fp32 accumulate).
//
// K is walked in slabs of 64.  Each slab of A (BM x 64) and B (64 x BN) is
// staged through LDS, double-buffered: the global loads of slab k+1 are in
// flight while slab k feeds the MFMAs.  MFMA operands want K contiguous per
// lane, so A is stored as is and B is stored transposed ([n][k]); the
// transpose is done in registers, one 8 x 8 block per thread.  LDS rows are
// 128 bytes with their 16-byte chunks XOR-swizzled so that both the staging
// writes and the operand reads are free of bank conflicts.
//
// The K tail (K % 64) is zero-filled (K % 8 == 0 keeps 16-byte rows whole).
//
// Epilogue: the MFMA is issued with the B fragment as its first operand, so
// each lane ends up holding 4 consecutive N values of one output row; they
// are rounded to bf16 (nearest even) and stored 8 bytes at a time.  Then the
// workgroup synchronises and one thread publishes the block's tile flags.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "flags.h"
#include "tile_order.h"

namespace entwine {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  int64_t lda, ldb, ldc;
  int M, N, K, P, order;
  int* flags;       // one per global 128 x 128 tile, row-major; null = no publish
  uint32_t epoch;
};

template <int BM_, int BN_>
struct GemmShape {
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int BK = 64;
  static constexpr int THREADS = 256;
  static constexpr int WM = BM / 2, WN = BN / 2;     // wave sub-block
  static constexpr int FM = WM / 32, FN = WN / 32;   // 32 x 32 MFMA blocks per wave
  static constexpr int A_BYTES = BM * BK * 2;
  static constexpr int B_BYTES = BN * BK * 2;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS_BYTES = 2 * STAGE;
  static constexpr int A_CHUNKS = BM * (BK / 8) / THREADS;   // 16-byte chunks per thread
  static constexpr int B_THREADS = BN;                       // threads owning an 8 x 8 block
  static_assert(BM % 128 == 0 && BN % 128 == 0, "blocks are whole 128 x 128 tiles");
};

// Byte offset of 16-byte chunk kc (0..7) of LDS row `row` (128-byte rows).
__device__ __forceinline__ int lds_off(int row, int kc) {
  return row * 128 + (((kc ^ row ^ (row >> 3)) & 7) << 4);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2_t f = {lo, hi};
  bf16x2_t b = __builtin_convertvector(f, bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

template <int BM, int BN>
__global__ __launch_bounds__(256) void gemm_producer(GemmArgs a) {
  using S = GemmShape<BM, BN>;
  extern __shared__ __attribute__((aligned(16))) char smem[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const BlockGrid grid = make_grid(a.M, a.N, a.P, BM, BN);
  const BlockPos bp = block_of_position(a.order, blockIdx.x, grid);
  const int row0 = bp.mb * BM;
  const int col0 = bp.nb * BN;
  const int K = a.K;
  const int nk = (K + S::BK - 1) / S::BK;

  f32x16_t acc[S::FM][S::FN];
#pragma unroll
  for (int i = 0; i < S::FM; ++i)
#pragma unroll
    for (int j = 0; j < S::FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  u32x4_t ra[S::A_CHUNKS];
  u32x4_t rb[8];
  const bool b_owner = tid < S::B_THREADS;
  const int b_nc = tid % (BN / 8);   // 8-column group of the thread's 8 x 8 block
  const int b_kg = tid / (BN / 8);   // 8-row (K) group

  const uint16_t* Ablk = a.A + static_cast<int64_t>(row0) * a.lda;
  const uint16_t* Bblk = a.B + col0 + b_nc * 8;

  auto gload = [&](int kt) {
    const int k0 = kt * S::BK;
#pragma unroll
    for (int i = 0; i < S::A_CHUNKS; ++i) {
      const int ci = tid + S::THREADS * i;
      const int r = ci >> 3, kc = ci & 7;
      const int k = k0 + kc * 8;
      ra[i] = (k < K) ? *reinterpret_cast<const u32x4_t*>(Ablk + static_cast<int64_t>(r) * a.lda + k)
                      : u32x4_t{0, 0, 0, 0};
    }
    if (b_owner) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = k0 + b_kg * 8 + j;
        rb[j] = (k < K) ? *reinterpret_cast<const u32x4_t*>(Bblk + static_cast<int64_t>(k) * a.ldb)
                        : u32x4_t{0, 0, 0, 0};
      }
    }
  };

  auto lstore = [&](int stage) {
    char* As = smem + stage * S::STAGE;
    char* Bs = As + S::A_BYTES;
#pragma unroll
    for (int i = 0; i < S::A_CHUNKS; ++i) {
      const int ci = tid + S::THREADS * i;
      *reinterpret_cast<u32x4_t*>(As + lds_off(ci >> 3, ci & 7)) = ra[i];
    }
    if (b_owner) {
      // rb[j] holds B[k = 8 kg + j][n = 8 nc .. 8 nc + 7]; column i of that
      // 8 x 8 block becomes row n = 8 nc + i of the transposed slab.
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        u32x4_t t;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t x = rb[2 * q][i >> 1];
          const uint32_t y = rb[2 * q + 1][i >> 1];
          t[q] = (i & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
        }
        *reinterpret_cast<u32x4_t*>(Bs + lds_off(b_nc * 8 + i, b_kg)) = t;
      }
    }
  };

  auto compute = [&](int stage) {
    const char* As = smem + stage * S::STAGE;
    const char* Bs = As + S::A_BYTES;
#pragma unroll
    for (int kk = 0; kk < S::BK / 16; ++kk) {
      const int kc = kk * 2 + (lane >> 5);
      bf16x8_t af[S::FM], bfr[S::FN];
#pragma unroll
      for (int i = 0; i < S::FM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(As + lds_off(wm * S::WM + i * 32 + (lane & 31), kc));
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t*>(Bs + lds_off(wn * S::WN + j * 32 + (lane & 31), kc));
#pragma unroll
      for (int i = 0; i < S::FM; ++i)
#pragma unroll
        for (int j = 0; j < S::FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
  };

  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    compute(cur);
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds D[n][m] for m = lane % 32 and
  // n = 8 (v / 4) + 4 (lane / 32) + v % 4, v = 0..15 (D = C^T).
#pragma unroll
  for (int i = 0; i < S::FM; ++i) {
    const int m = row0 + wm * S::WM + i * 32 + (lane & 31);
    uint16_t* crow = a.C + static_cast<int64_t>(m) * a.ldc;
#pragma unroll
    for (int j = 0; j < S::FN; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = col0 + wn * S::WN + j * 32 + g * 8 + (lane >> 5) * 4;
        u32x2_t w;
        w[0] = pack_bf16x2(acc[i][j][4 * g + 0], acc[i][j][4 * g + 1]);
        w[1] = pack_bf16x2(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
        *reinterpret_cast<u32x2_t*>(crow + n) = w;
      }
    }
  }

  if (a.flags != nullptr) {
    __syncthreads();
    if (tid == 0) {
      const int tiles_n = a.N / kTile;
#pragma unroll
      for (int ti = 0; ti < BM / kTile; ++ti)
#pragma unroll
        for (int tj = 0; tj < BN / kTile; ++tj)
          publish_release(a.flags + (bp.mb * (BM / kTile) + ti) * tiles_n + bp.nb * (BN / kTile) + tj,
                          a.epoch);
    }
  }
}

}  // namespace entwine
