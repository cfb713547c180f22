// gemm_producer.h - the producer: a bf16 MFMA GEMM for gfx950 whose
// workgroups take their output blocks in a chosen traversal order and
// publish a ready flag per 128 x 128 tile (paper Sections 3.1 and 4.2).
//
// One workgroup computes a BM x BN block of C = A B (A: M x K, B: K x N, both
// row-major bf16) with 4 waves in a 2 x 2 arrangement; each wave owns a
// (BM/2) x (BN/2) sub-block held as 32 x 32 MFMA accumulators
// (v_mfma_f32_32x32x16_bf16: fp32 accumulate, 16 K per instruction).
//
// Data path per K-slab of 32:
//  * global -> LDS with direct-to-LDS loads (global_load_lds_dwordx4): each
//    instruction moves 64 lanes x 16 bytes into 1 KB of contiguous LDS, no
//    registers involved.  A slab lives in one of 4 LDS stages; the loads for
//    slab k+3 are issued while slab k is being multiplied.
//  * LDS layouts are chosen for conflict-free operand reads, and realised by
//    permuting which global 16-byte chunk each lane fetches:
//      A stage: [BM rows][32 k] (64-byte rows), chunk c of row r stored at
//               chunk c ^ ((r >> 2) & 3);
//      B stage: [32 k][BN n] (row-major, as in memory), chunk c of row k
//               stored at chunk c ^ (4 (k & 3)).
//  * A operands: one ds_read_b128 per 32 x 16 fragment (8 consecutive k per
//    lane).  B operands: the MFMA wants 8 consecutive k of one column per
//    lane, while B is row-major; gfx950's ds_read_b64_tr_b16 transposes
//    4 x 16 blocks across each group of 16 lanes (lane i receives element
//    i % 4 of the 8 bytes addressed by lane 4e + i / 4, for e = 0..3), so two
//    such reads build one fragment with no register shuffles.
//  * Operand fragments of slab k+1 are read from LDS before the MFMAs of
//    slab k are issued (double-buffered in registers).
// The K tail (K % 32) is handled without branches: lanes whose 16-byte chunk
// lies beyond K fetch from a zero page instead.
//
// Epilogue: the MFMA is issued with the B fragment as its first operand, so
// each lane ends up holding 4 consecutive N values of one output row; they
// are rounded to bf16 (nearest even) and stored 8 bytes at a time.  Then the
// workgroup synchronises and one thread publishes the block's tile flags.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "flags.h"
#include "tile_order.h"

namespace entwine {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  const uint16_t* zeros;  // >= 16 readable bytes of zeros (K-tail fill)
  int64_t lda, ldb, ldc;
  int M, N, K, P, order, group_m;
  int* flags;             // one per global 128 x 128 tile, row-major; null = no publish
  uint32_t epoch;
};

template <int BM_, int BN_>
struct GemmShape {
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int BK = 32;
  static constexpr int THREADS = 256;
  static constexpr int STAGES = 4;
  static constexpr int WM = BM / 2, WN = BN / 2;     // wave sub-block
  static constexpr int FM = WM / 32, FN = WN / 32;   // 32 x 32 MFMA blocks per wave
  static constexpr int A_STAGE = BM * BK * 2;        // bytes
  static constexpr int B_STAGE = BK * BN * 2;
  static constexpr int A_DMA = A_STAGE / 1024 / 4;   // 1 KB loads per wave per slab
  static constexpr int B_DMA = B_STAGE / 1024 / 4;
  static constexpr int DMA = A_DMA + B_DMA;
  static constexpr int B_ROW = BN * 2;               // bytes per LDS row of B
  static constexpr int B_CPR = BN / 8;               // 16-byte chunks per B row
  static constexpr int C_BYTES = 32 * 1024;           // epilogue staging, 8 KB per wave
  static constexpr int LDS_BYTES = STAGES * (A_STAGE + B_STAGE) + C_BYTES;
  static_assert(BM % 128 == 0 && BN % 128 == 0, "blocks are whole 128 x 128 tiles");
};

template <int V>
using IC = std::integral_constant<int, V>;

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  // C-style cast: generic -> LDS address space (no C++ cast performs it).
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 64 lanes x 16 bytes from `src` (per lane) into LDS [lds, lds + 1 KB).  The
// load is hidden from the compiler's wait tracking; callers wait with
// wait_vm<N>() before a barrier that precedes any read of the data.
// The compiler does not insert hazard wait states for operands of inline
// asm, so the asm carries them: GFX9 needs 1 wait state between a scalar
// write of M0 and an LDS-DMA load reading it.
__device__ __forceinline__ void dma16(const void* src, uint32_t lds) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(lds) : "memory");
}

// Same, addressing with a wave-uniform 64-bit base and a 32-bit per-lane
// byte offset (the saddr form): no per-lane 64-bit address arithmetic.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
  return reinterpret_cast<const void*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// The base usually arrives through v_readfirstlane (a VALU write of an
// SGPR); GFX9 needs 5 wait states between that and a VMEM instruction
// reading the SGPR, which also covers the M0 wait state above.
__device__ __forceinline__ void dma16_s(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_nop 4\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(uniform_ptr(base)), "{m0}"(lds)
               : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2_t f = {lo, hi};
  bf16x2_t b = __builtin_convertvector(f, bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ bf16x4_t ds_read_tr(const char* p) {
  typedef __attribute__((address_space(3))) i16x4_t lds_i16x4;
  i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(__attribute__((address_space(3))) char*)p);
  return __builtin_bit_cast(bf16x4_t, v);
}

template <int BM, int BN>
__global__ __launch_bounds__(256) void gemm_producer(GemmArgs a) {
  using S = GemmShape<BM, BN>;
  // LDS: 4 A stages, 4 B stages, then a C staging area (8 KB per wave).
  __shared__ __attribute__((aligned(1024))) char smem[S::LDS_BYTES];
  char* const sA = smem;
  char* const sB = smem + 4 * S::A_STAGE;
  char* const sC = smem + 4 * (S::A_STAGE + S::B_STAGE);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // ---- work of this workgroup: logical positions p = w, w + G, w + 2G, ...
  // Positions are taken in increasing order, so production time follows the
  // logical order of the traversal; all its K-slabs form one stream, so the
  // loads of the next block start while the current block finishes.
  const BlockGrid grid = make_grid(a.M, a.N, a.P, BM, BN, a.group_m);
  const int nblk = grid.MB * grid.NB;
  const int G = gridDim.x, w = blockIdx.x;
  const int mine = w < nblk ? (nblk - 1 - w) / G + 1 : 0;
  const int K = a.K;
  const int nk = (K + S::BK - 1) / S::BK;
  const int total = mine * nk;
  if (total == 0) return;

  // ---- per-lane DMA sources: byte offsets inside a block, and their K
  uint32_t a_off[S::A_DMA], b_off[S::B_DMA];
  int a_k[S::A_DMA], b_k[S::B_DMA];
#pragma unroll
  for (int i = 0; i < S::A_DMA; ++i) {
    const int r = (wave * S::A_DMA + i) * 16 + (lane >> 2);
    const int lc = (lane & 3) ^ ((r >> 2) & 3);
    a_off[i] = static_cast<uint32_t>((r * a.lda + lc * 8) * 2);
    a_k[i] = lc * 8;
  }
#pragma unroll
  for (int i = 0; i < S::B_DMA; ++i) {
    const int fc = (wave * S::B_DMA + i) * 64 + lane;
    const int r = fc / S::B_CPR;
    const int lc = (fc % S::B_CPR) ^ (4 * (r & 3));
    b_off[i] = static_cast<uint32_t>((r * a.ldb + lc * 8) * 2);
    b_k[i] = r;
  }

  // DMA cursor: the next slab of the stream to load (block d_lb, slab d_kt).
  int d_g = 0, d_kt = 0, d_lb = 0;
  auto uniform_block = [&](int p) {
    BlockPos b = block_of_position(a.order, p, grid);
    b.mb = __builtin_amdgcn_readfirstlane(b.mb);
    b.nb = __builtin_amdgcn_readfirstlane(b.nb);
    return b;
  };
  BlockPos d_bp = uniform_block(w);
  struct DmaSlab {
    const char* Ab;
    const char* Bb;
    uint32_t la, lb;
    int k0;
    bool whole;   // the slab lies entirely inside K
  };
  auto dma_prep = [&]() {
    DmaSlab d;
    const int st = d_g & 3;
    d.k0 = d_kt * S::BK;
    d.Ab = reinterpret_cast<const char*>(a.A + static_cast<int64_t>(d_bp.mb * BM) * a.lda + d.k0);
    d.Bb = reinterpret_cast<const char*>(a.B + static_cast<int64_t>(d.k0) * a.ldb + d_bp.nb * BN);
    d.la = lds_u32(sA + st * S::A_STAGE + wave * S::A_DMA * 1024);
    d.lb = lds_u32(sB + st * S::B_STAGE + wave * S::B_DMA * 1024);
    d.whole = d.k0 + S::BK <= K;
    return d;
  };
  // Load i of a whole slab (i < A_DMA: A, else B).
  auto dma_issue = [&](const DmaSlab& d, int i) {
    if (i < S::A_DMA) dma16_s(d.Ab, a_off[i], d.la + i * 1024);
    else dma16_s(d.Bb, b_off[i - S::A_DMA], d.lb + (i - S::A_DMA) * 1024);
  };
  // A slab that crosses K: lanes past K read zeros.
  auto dma_tail = [&](const DmaSlab& d) {
#pragma unroll
    for (int i = 0; i < S::A_DMA; ++i)
      dma16((d.k0 + a_k[i] < K) ? static_cast<const void*>(d.Ab + a_off[i]) : static_cast<const void*>(a.zeros),
            d.la + i * 1024);
#pragma unroll
    for (int i = 0; i < S::B_DMA; ++i)
      dma16((d.k0 + b_k[i] < K) ? static_cast<const void*>(d.Bb + b_off[i]) : static_cast<const void*>(a.zeros),
            d.lb + i * 1024);
  };
  auto dma_advance = [&]() {
    ++d_g;
    if (++d_kt == nk) {
      d_kt = 0;
      if (++d_lb < mine) d_bp = uniform_block(w + d_lb * G);
    }
  };
  auto dma_next = [&]() {   // a whole slab, not interleaved (prologue)
    const DmaSlab d = dma_prep();
    if (d.whole) {
#pragma unroll
      for (int i = 0; i < S::DMA; ++i) dma_issue(d, i);
    } else {
      dma_tail(d);
    }
    dma_advance();
  };

  // ---- per-lane LDS read offsets (bytes, relative to a stage)
  // A fragment (rows wm*WM + i*32 + lane%32, 8 k per lane at 16 kk + 8 (lane/32)).
  const int a_row = wm * S::WM + (lane & 31);
  const int a_rd0 = a_row * 64 + (((lane >> 5) ^ ((a_row >> 2) & 3)) << 4);
  const int a_rd1 = a_row * 64 + (((2 + (lane >> 5)) ^ ((a_row >> 2) & 3)) << 4);
  // B fragment via transpose reads: lane = 16 g + i; reads row
  // k = 16 kk + 8 (g / 2) + 4 h + i / 4, columns n .. n+3 with
  // n = wn*WN + 32 j + 16 (g % 2) + 4 (i % 4).
  const int b_kq = (lane >> 2) & 3;                       // k & 3 of the row read
  const int b_row = (8 * (lane >> 5) + b_kq) * S::B_ROW;  // + (16 kk + 4 h) * B_ROW
  int b_col[S::FN];
#pragma unroll
  for (int j = 0; j < S::FN; ++j) {
    const int n = wn * S::WN + 32 * j + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    b_col[j] = (((n >> 3) ^ (4 * b_kq)) << 4) + ((n & 7) << 1);
  }

  // Fragments of one K-half (16 k) of a slab.
  struct Frags {
    bf16x8_t a[S::FM];
    bf16x8_t b[S::FN];
  };
  constexpr int NREAD = S::FM + S::FN;       // LDS read ops per half
  // Read op r of a half: r < FM reads A fragment r; the others read both
  // 4-k halves of one B fragment.
  auto read_one = [&](Frags& f, int st, int kk, int r) {
    if (r < S::FM) {
      f.a[r] = *reinterpret_cast<const bf16x8_t*>(sA + st * S::A_STAGE + (kk ? a_rd1 : a_rd0) + r * 32 * 64);
    } else {
      const int j = r - S::FM;
      const char* p = sB + st * S::B_STAGE + b_row + 16 * kk * S::B_ROW + b_col[j];
      const bf16x4_t lo = ds_read_tr(p);
      const bf16x4_t hi = ds_read_tr(p + 4 * S::B_ROW);
      f.b[j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  };
  auto read_half = [&](Frags& f, int st, int kk) {
#pragma unroll
    for (int r = 0; r < NREAD; ++r) read_one(f, st, kk, r);
  };

  f32x16_t acc[S::FM][S::FN];
  constexpr int NMF = S::FM * S::FN;         // MFMAs per half
  auto mfma_one = [&](const Frags& f, int m) {
    const int i = m / S::FN, j = m % S::FN;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[j], f.a[i], acc[i][j], 0, 0, 0);
  };

  // One slab g of the stream; on entry X holds the first K-half of slab g.
  //  phase A: the MFMAs of X, with the LDS reads of the second half (Y)
  //           spread between them;
  //  then:    own loads of slab g+1 done, barrier (slab g+1 visible to the
  //           whole workgroup, and the stage of slab g-1 free again);
  //  phase B: the MFMAs of Y, with the reads of slab g+1's first half (X)
  //           and the loads of slab g+3 (into the freed stage) spread
  //           between them.
  // sched_barrier pins the interleaving so the matrix core always has the
  // next MFMA queued while the other instructions issue.
  Frags X, Y;
  auto step = [&](int g) {
    const int st = g & 3;
#pragma unroll
    for (int m = 0; m < NMF; ++m) {
      mfma_one(X, m);
#pragma unroll
      for (int r = m * NREAD / NMF; r < (m + 1) * NREAD / NMF; ++r) read_one(Y, st, 1, r);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (g + 2 < total) wait_vm<S::DMA>();
    else wait_vm<0>();
    __syncthreads();
    // The next half is always read (past the end of the stream it is a
    // harmless read of a free stage); the loads of slab g+3 are skipped past
    // the end, and a slab that crosses K is issued before the MFMAs.
    const int nst = (g + 1) & 3;
    const bool ld = g + 3 < total;
    const DmaSlab d = dma_prep();
    const bool ld_whole = ld && d.whole;
    if (ld && !d.whole) dma_tail(d);
    constexpr int NOPS = NREAD + S::DMA;
#pragma unroll
    for (int m = 0; m < NMF; ++m) {
      mfma_one(Y, m);
#pragma unroll
      for (int o = m * NOPS / NMF; o < (m + 1) * NOPS / NMF; ++o) {
        if (o < NREAD) read_one(X, nst, 0, o);
        else if (ld_whole) dma_issue(d, o - NREAD);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (ld) dma_advance();
  };

  dma_next();
  if (total > 1) dma_next();
  if (total > 2) dma_next();
  if (total > 2) wait_vm<2 * S::DMA>();
  else if (total > 1) wait_vm<S::DMA>();
  else wait_vm<0>();
  __syncthreads();
  read_half(X, 0, 0);

  constexpr int CPR = S::WN / 8;                 // 16-byte chunks per staged row
  constexpr int ROWB = S::WN * 2;                // bytes per staged row
  char* const cst = sC + wave * (32 * ROWB);     // 32 rows per wave
  static_assert(4 * 32 * ROWB <= S::C_BYTES, "C staging fits");

  int g = 0;
  for (int lb = 0; lb < mine; ++lb) {
    const BlockPos bp = block_of_position(a.order, w + lb * G, grid);
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
    for (int kt = 0; kt < nk; ++kt) step(g++);

    // ---- epilogue.  Lane holds D[n][m] for m = lane % 32 and
    // n = 8 (v / 4) + 4 (lane / 32) + v % 4, v = 0..15 (D = C^T): 4
    // consecutive columns of one row per group of 4 registers.  Each wave
    // stages 32 rows of its (BM/2) x (BN/2) sub-block at a time in its own
    // LDS area (16-byte chunks XOR-swizzled by row), then stores whole rows
    // with 16-byte lanes, so every store instruction writes full 128-byte
    // lines.  The stores are non-temporal: the partial is read once, by the
    // reducer, and streaming it past L2 leaves little dirty data for the
    // release fence to write back.
    uint16_t* cblk = a.C + static_cast<int64_t>(bp.mb * BM + wm * S::WM) * a.ldc + bp.nb * BN + wn * S::WN;
#pragma unroll
    for (int i = 0; i < S::FM; ++i) {
      const int r = lane & 31;
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c = 4 * j + q;               // chunk of columns 32 j + 8 q .. + 7
          u32x2_t v2;
          v2[0] = pack_bf16x2(acc[i][j][4 * q + 0], acc[i][j][4 * q + 1]);
          v2[1] = pack_bf16x2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
          *reinterpret_cast<u32x2_t*>(cst + r * ROWB + ((c ^ (r % CPR)) << 4) + (lane >> 5) * 8) = v2;
        }
      // The staged rows are private to the wave; LDS operations of one wave
      // complete in order, so the reads below see the writes above.
      constexpr int RPI = 64 / CPR;              // rows per store instruction
#pragma unroll
      for (int r0 = 0; r0 < 32; r0 += RPI) {
        const int rr = r0 + lane / CPR, c = lane % CPR;
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(cst + rr * ROWB + ((c ^ (rr % CPR)) << 4));
        __builtin_nontemporal_store(
            v, reinterpret_cast<u32x4_t*>(cblk + static_cast<int64_t>(i * 32 + rr) * a.ldc + c * 8));
      }
    }

    if (a.flags != nullptr) {
      __syncthreads();
      if (tid == 0) {
        const int tiles_n = a.N / kTile;
        release_fence();
#pragma unroll
        for (int ti = 0; ti < BM / kTile; ++ti)
#pragma unroll
          for (int tj = 0; tj < BN / kTile; ++tj)
            publish_relaxed(a.flags + (bp.mb * (BM / kTile) + ti) * tiles_n + bp.nb * (BN / kTile) + tj,
                            a.epoch);
      }
    }
  }
}

}  // namespace entwine
