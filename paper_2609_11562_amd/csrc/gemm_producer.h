// gemm_producer.h - the producer: a bf16 MFMA GEMM for gfx950 whose
// workgroups take their output blocks in a chosen traversal order and
// publish a ready flag per 128 x 128 tile (paper Sections 3.1 and 4.2).
//
// One workgroup computes BM x BN blocks of C = A B (A: M x K, B: K x N, both
// row-major bf16) with 4 waves in a 2 x 2 arrangement; each wave owns a
// (BM/2) x (BN/2) sub-block held as 32 x 32 MFMA accumulators
// (v_mfma_f32_32x32x16_bf16: fp32 accumulate, 16 K per instruction).  The
// kernel is persistent: workgroup w of G takes logical positions w, w + G,
// w + 2G, ... and streams all their K-slabs as one sequence.
//
// Data path, per K-slab of 32 (two MFMA K-steps of 16):
//  * global -> LDS with direct-to-LDS loads (global_load_lds_dwordx4): each
//    instruction moves 64 lanes x 16 bytes into 1 KB of contiguous LDS, no
//    registers involved.  Slabs rotate through 4 LDS stages.
//  * The texture path of a CU accepts roughly one such load per 16 cycles,
//    so a burst of loads stalls the wave that issues them (and with it the
//    matrix core).  Each wave's loads of a slab are therefore spread evenly
//    over two K-steps of MFMAs: slab s + 3 is loaded, half in the last K-step
//    of slab s - 1 and half in the first K-step of slab s, into the stage
//    that slab s - 1 has just released.  A slab's loads are issued at least
//    two slabs before it is read.
//  * One workgroup barrier per slab, before its last K-step: by then every
//    wave has read all of the slab's operands into registers (its stage is
//    free) and its own loads of the next slab have landed.
//  * LDS layouts are chosen for conflict-free operand reads, and realised by
//    permuting which global 16-byte chunk each lane fetches:
//      A stage: [BM rows][32 k] (64-byte rows), chunk c of row r stored at
//               chunk c ^ a_swizzle(r) (below);
//      B stage: [32 k][BN n] (row-major, as in memory), chunk c of row k
//               stored at chunk c ^ (4 (k & 3)).
//  * A operands: one ds_read_b128 per 32 x 16 fragment (8 consecutive k per
//    lane).  B operands: the MFMA wants 8 consecutive k of one column per
//    lane, while B is row-major; gfx950's ds_read_b64_tr_b16 transposes
//    4 x 16 blocks across each group of 16 lanes (lane i receives element
//    i % 4 of the 8 bytes addressed by lane 4e + i / 4, for e = 0..3), so two
//    such reads build one fragment with no register shuffles.
//  * Operand fragments of the next K-step are read from LDS between the
//    first MFMAs of the current one (two register buffers), in the order the
//    MFMAs consume them.
// The K tail (K % 32) goes through the same loads with a per-lane address:
// lanes whose 16-byte chunk lies beyond K fetch from a zero page instead.
//
// Epilogue: the MFMA is issued with the B fragment as its first operand, so
// each lane ends up holding 4 consecutive N values of one output row; they
// are rounded to bf16 (nearest even), staged through LDS and stored as whole
// rows.  Then the workgroup synchronises and one thread publishes the
// block's tile flags after a release fence.
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
  int release_blocks;     // publish after every g blocks (g >= 1), only after the last (g = -1), or
                          // by group: -2 a partition's tiles once all are stored, -3 the whole output's
  int store_mode;         // tile stores: 0 write-through; 1 non-temporal, 2 write-back (both written
                          // back from L2 at the release)
  unsigned long long* group_ctr;   // release groups: tiles stored, per partition (P) then the output (1);
                                   // a multiple of the group's tile count between calls
  unsigned int* take_ctr;  // fused launch: the reduction task counter, first taken during the last epilogue
};

constexpr int kReleasePartition = -2;
constexpr int kReleaseOutput = -3;

template <int BM_, int BN_>
struct GemmShape {
  static constexpr int BM = BM_, BN = BN_;
  static constexpr int BK = 32;                      // K per slab
  static constexpr int Q = BK / 16;                  // MFMA K-steps per slab
  static constexpr int THREADS = 256;
  static constexpr int WM = BM / 2, WN = BN / 2;     // wave sub-block
  static constexpr int FM = WM / 32, FN = WN / 32;   // 32 x 32 MFMA blocks per wave
  static constexpr int A_ROW = BK * 2;               // bytes per LDS row of A
  static constexpr int B_ROW = BN * 2;               // bytes per LDS row of B
  static constexpr int A_STAGE = BM * A_ROW;
  static constexpr int B_STAGE = BK * B_ROW;
  static constexpr int STAGE = A_STAGE + B_STAGE;    // one slab: A part, then B part
  static constexpr int STAGES = 4;
  static constexpr int ROWB = WN * 2;                // bytes per staged C row
  static constexpr int C_BYTES = 4 * 32 * ROWB;      // epilogue staging, 32 rows per wave
  static constexpr int LDS_BYTES = STAGES * STAGE + C_BYTES;
  static constexpr int A_DMA = A_STAGE / 1024 / 4;   // 1 KB loads per wave per slab
  static constexpr int B_DMA = B_STAGE / 1024 / 4;
  static constexpr int DMA = A_DMA + B_DMA;
  static constexpr int DH = DMA / 2;                 // loads per half slab
  static constexpr int B_CPR = BN / 8;               // 16-byte chunks per B row
  static_assert(BM % 128 == 0 && BN % 128 == 0, "blocks are whole 128 x 128 tiles");
  static_assert(Q == 2 && DMA % 2 == 0, "two K-steps per slab, loads split in halves");
  static_assert(LDS_BYTES <= 160 * 1024, "gfx950 LDS per workgroup");
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

// The base may arrive through v_readfirstlane (a VALU write of an SGPR), and
// GFX9 needs 5 wait states between that and a VMEM instruction reading the
// SGPR.  The asm therefore copies the base into fresh SGPRs with a scalar
// move (a scalar write is not subject to that rule) and loads through the
// copy; the move also provides the wait state after the write of M0.
__device__ __forceinline__ void dma16_s(const void* base, uint32_t off, uint32_t lds) {
  uint64_t tmp;
  asm volatile("s_mov_b64 %0, %2\n\tglobal_load_lds_dwordx4 %1, %0"
               : "=&s"(tmp)
               : "v"(off), "s"(uniform_ptr(base)), "{m0}"(lds)
               : "memory");
}

// 16-byte chunk permutation of A stage row r.  An A fragment read
// (ds_read_b128) puts lanes 0-31 (and 32-63) on 32 consecutive rows at one
// logical chunk.  On gfx950 the LDS bank-conflict counter (a probe of this
// exact pattern) reads zero for XOR masks (r >> 2) & 3, (r >> 3) & 3 and
// (r ^ (r >> 2)) & 3, and 2-way conflicts for ((r >> 1) ^ (r >> 3)) & 3,
// (r >> 1) & 3 and ((r >> 2) ^ (r >> 4)) & 3 (4-way unpermuted).
// (r ^ (r >> 2)) & 3 is the one of the three that is also conflict-free in
// the textbook bank models (8 lanes over 32 banks, 16 lanes over 64).
__device__ __forceinline__ int a_swizzle(int r) { return (r ^ (r >> 2)) & 3; }

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Orders LDS accesses between the lanes of one wave (release, wave barrier,
// acquire at wavefront scope).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
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

template <int N>
__device__ __forceinline__ void wait_slabs_le(int n) {
  // Wait until at most n slabs (n * N loads of this wave) are outstanding.
  switch (n) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<N>(); break;
    default: wait_vm<2 * N>(); break;
  }
}

template <int D, int DH>
__device__ __forceinline__ void wait_loads_le(int n) {
  // Wait until at most n loads of this wave are outstanding, n a multiple of
  // DH no larger than 2 D + DH.
  if (n >= 2 * D + DH) wait_vm<2 * D + DH>();
  else if (n >= 2 * D) wait_vm<2 * D>();
  else if (n >= D + DH) wait_vm<D + DH>();
  else if (n >= D) wait_vm<D>();
  else if (n >= DH) wait_vm<DH>();
  else wait_vm<0>();
}

// Store 16 bytes with system scope (sc0 sc1): the data is written through
// the L2 instead of being left dirty in it, so the release fence that
// publishes a tile has little to write back.  The trailing wait state covers
// the hazard of a VALU write to the store's data registers right after a
// store of more than 8 bytes (the compiler does not insert it for asm).
__device__ __forceinline__ void store16_wt(void* dst, u32x4_t v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc0 sc1\n\ts_nop 0" ::"v"(dst), "v"(v) : "memory");
}

// TAIL: K % 32 != 0.  Without a tail every slab is whole, so the loads are
// issued unconditionally: past the end of the stream they re-read the last
// slab (valid memory) into the stage that is free at that point, which no
// real slab uses again; they are drained before the kernel ends.
// The producer role of workgroup w of G; `smem` is GemmShape::LDS_BYTES of
// LDS, 1 KB aligned.  Used by gemm_producer and by the single-launch fused
// kernel, whose first G workgroups are producers.  Returns, in thread 0 when
// a.take_ctr is set and the workgroup had blocks, the reduction task it took
// at the start of its last epilogue (the atomic's round trip then overlaps
// the epilogue); ~0u otherwise.
template <int BM, int BN, bool TAIL>
__device__ __forceinline__ unsigned int producer_body(const GemmArgs& a, const int w, const int G, char* smem) {
  using S = GemmShape<BM, BN>;
  constexpr int NS = S::STAGES;
  constexpr int D = S::DMA, DH = S::DH;
  static_assert(2 * D + DH < 64, "vmcnt range");

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
  const int mine = w < nblk ? (nblk - 1 - w) / G + 1 : 0;
  const int K = a.K;
  const int nk = (K + S::BK - 1) / S::BK;
  const int total = mine * nk;
  if (total == 0) return ~0u;

  // ---- per-lane load sources: byte offsets inside a block, and their K.
  // A: one load fills 16 rows of 64 bytes; lane -> row lane / 4, stored
  // chunk lane % 4, which holds logical chunk (lane % 4) ^ sw(row).
  // B: one load fills 1 KB of consecutive [k][n] rows.
  uint32_t a_off[S::A_DMA], b_off[S::B_DMA];
  int a_k[S::A_DMA], b_k[S::B_DMA];
#pragma unroll
  for (int i = 0; i < S::A_DMA; ++i) {
    const int r = (wave * S::A_DMA + i) * 16 + (lane >> 2);
    const int lc = (lane & 3) ^ a_swizzle(r);
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

  // ---- load cursor: the slab being loaded (block d_lb, slab d_kt of it),
  // with wave-uniform base addresses advanced incrementally.
  auto uniform_block = [&](int p) {
    BlockPos b = block_of_position(a.order, p, grid);
    b.mb = __builtin_amdgcn_readfirstlane(b.mb);
    b.nb = __builtin_amdgcn_readfirstlane(b.nb);
    return b;
  };
  auto a_base = [&](const BlockPos& b) {
    return reinterpret_cast<const char*>(a.A + static_cast<int64_t>(b.mb * BM) * a.lda);
  };
  auto b_base = [&](const BlockPos& b) { return reinterpret_cast<const char*>(a.B + b.nb * BN); };
  int d_g = 0, d_kt = 0, d_lb = 0;
  BlockPos d_bp = uniform_block(w);
  const char* dA = a_base(d_bp);
  const char* dB = b_base(d_bp);
  const int64_t b_step = static_cast<int64_t>(S::BK) * a.ldb * 2;   // bytes per slab of B
  static_assert((NS & (NS - 1)) == 0, "stage index by mask");
  auto st_base = [&](int g) { return smem + (g & (NS - 1)) * S::STAGE; };
  auto la_of = [&](int g) { return lds_u32(st_base(g) + wave * S::A_DMA * 1024); };
  auto lb_of = [&](int g) { return lds_u32(st_base(g) + S::A_STAGE + wave * S::B_DMA * 1024); };
  auto d_whole = [&]() { return (d_kt + 1) * S::BK <= K; };
  // Load o (0 <= o < D) of the cursor's slab, which lies inside K: o < A_DMA
  // from A, else from B.
  auto dma_issue = [&](uint32_t la, uint32_t lb, int o) {
    if (o < S::A_DMA) dma16_s(dA, a_off[o], la + o * 1024);
    else dma16_s(dB, b_off[o - S::A_DMA], lb + (o - S::A_DMA) * 1024);
  };
  // Loads [o0, o1) of the cursor's slab, which crosses K: lanes past K read zeros.
  auto dma_tail = [&](uint32_t la, uint32_t lb, int o0, int o1) {
    const int k0 = d_kt * S::BK;
#pragma unroll
    for (int o = 0; o < D; ++o) {
      if (o < o0 || o >= o1) continue;
      if (o < S::A_DMA) {
        dma16((k0 + a_k[o] < K) ? static_cast<const void*>(dA + a_off[o]) : static_cast<const void*>(a.zeros),
              la + o * 1024);
      } else {
        const int i = o - S::A_DMA;
        dma16((k0 + b_k[i] < K) ? static_cast<const void*>(dB + b_off[i]) : static_cast<const void*>(a.zeros),
              lb + i * 1024);
      }
    }
  };
  // Loads [o0, o1) of the cursor's slab, not interleaved with MFMAs.
  auto dma_range = [&](int o0, int o1) {
    const uint32_t la = la_of(d_g), lb = lb_of(d_g);
    if (!TAIL || d_whole()) {
#pragma unroll
      for (int o = 0; o < D; ++o)
        if (o >= o0 && o < o1) dma_issue(la, lb, o);
    } else {
      dma_tail(la, lb, o0, o1);
    }
  };
  // Past the last slab the cursor stays on it.
  auto dma_advance = [&]() {
    ++d_g;
    if (d_lb == mine) return;
    if (++d_kt == nk) {
      if (++d_lb < mine) {
        d_kt = 0;
        d_bp = uniform_block(w + d_lb * G);
        dA = a_base(d_bp);
        dB = b_base(d_bp);
      } else {
        d_kt = nk - 1;
      }
    } else {
      dA += S::BK * 2;
      dB += b_step;
    }
  };

  // ---- per-lane LDS read offsets (bytes, relative to a stage)
  // A fragment i of K-step q: rows wm*WM + 32 i + lane % 32, 8 consecutive k
  // at 16 q + 8 (lane / 32), i.e. logical chunk 2 q + lane / 32.
  const int a_row = wm * S::WM + (lane & 31);
  const int a_sw = a_swizzle(a_row);                      // same for a_row + 32 i
  int a_rd[S::Q];
#pragma unroll
  for (int q = 0; q < S::Q; ++q) a_rd[q] = a_row * S::A_ROW + (((2 * q + (lane >> 5)) ^ a_sw) << 4);
  // B fragment via transpose reads: lane = 16 g + i; reads row
  // k = 16 q + 8 (g / 2) + 4 h + i / 4, columns n .. n+3 with
  // n = wn*WN + 32 j + 16 (g % 2) + 4 (i % 4).
  const int b_kq = (lane >> 2) & 3;                       // k & 3 of the row read
  const int b_row = S::A_STAGE + (8 * (lane >> 5) + b_kq) * S::B_ROW;
  int b_col[S::FN];
#pragma unroll
  for (int j = 0; j < S::FN; ++j) {
    const int n = wn * S::WN + 32 * j + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    b_col[j] = (((n >> 3) ^ (4 * b_kq)) << 4) + ((n & 7) << 1);
  }

  // Fragments of one K-step.
  struct Frags {
    bf16x8_t a[S::FM];
    bf16x8_t b[S::FN];
  };
  constexpr int NREAD = S::FM + S::FN;       // LDS read ops per K-step
  // Read op r of K-step q, in the order the MFMAs consume the fragments:
  // A fragment 0, the B fragments, then the other A fragments.
  auto read_one = [&](Frags& f, const char* stg, int q, int r) {
    if (r == 0 || r > S::FN) {
      const int i = r == 0 ? 0 : r - S::FN;
      f.a[i] = *reinterpret_cast<const bf16x8_t*>(stg + a_rd[q] + i * 32 * S::A_ROW);
    } else {
      const int j = r - 1;
      const char* p = stg + b_row + 16 * q * S::B_ROW + b_col[j];
      const bf16x4_t lo = ds_read_tr(p);
      const bf16x4_t hi = ds_read_tr(p + 4 * S::B_ROW);
      f.b[j] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  };

  f32x16_t acc[S::FM][S::FN];
  constexpr int NMF = S::FM * S::FN;         // MFMAs per K-step
  auto mfma_one = [&](const Frags& f, int m) {
    const int i = m / S::FN, j = m % S::FN;
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[j], f.a[i], acc[i][j], 0, 0, 0);
  };
  // One K-step: the MFMAs of `cur`, with the NREAD reads of the next K-step
  // (into `nxt`, from stage `stg`, K-step qn) after the first NREAD MFMAs,
  // and loads [o0, o0 + DH) of the cursor's slab (when `ldw`) spread evenly
  // over all of them, each behind the second MFMA of its group (measured:
  // 2-3.5% fewer cycles per slab than behind the last).  Reading early leaves
  // the reads complete before the barrier or the next K-step needs them.
  // sched_barrier pins the interleaving so the matrix core always has the
  // next MFMA queued while the other instructions issue.
  static_assert(NREAD <= NMF, "one read op per MFMA at most");
  auto kstep = [&](const Frags& cur, Frags& nxt, const char* stg, int qn, bool ldw, uint32_t la, uint32_t lb,
                   int o0) {
#pragma unroll
    for (int m = 0; m < NMF; ++m) {
      mfma_one(cur, m);
      if (m < NREAD) read_one(nxt, stg, qn, m);
#pragma unroll
      for (int k = 0; k < DH; ++k)
        if (m == k * NMF / DH + (NMF / DH > 1 ? 1 : 0) && (!TAIL || ldw)) dma_issue(la, lb, o0 + k);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // One slab g of the stream; on entry X holds K-step 0 of slab g and the
  // cursor is at slab g + NS - 1 with its first half issued.
  //  K-step 0: MFMAs of X; reads of K-step 1 into Y; second half of the
  //            cursor's slab.
  //  then:     own loads of slab g+1 done, barrier: slab g+1 is visible to
  //            the workgroup, and every wave has read all of slab g.
  //  K-step 1: MFMAs of Y; reads of slab g+1's K-step 0 into X; first half
  //            of slab g + NS, into slab g's stage (free now).
  // Past the end of the stream no loads are issued and the reads of the next
  // K-step are harmless reads of a stage that is not used again.
  Frags X, Y;
  auto step = [&](int g) {
    {
      const bool ld = !TAIL || g + NS - 1 < total;
      const bool ldw = !TAIL || (ld && d_whole());
      const uint32_t la = la_of(d_g), lb = lb_of(d_g);
      if (TAIL && ld && !ldw) dma_tail(la, lb, DH, D);
      kstep(X, Y, st_base(g), 1, ldw, la, lb, DH);
      if (ld) dma_advance();
    }
    // slabs issued after g+1 that may still be in flight
    int after = NS - 2;
    if (TAIL && total - g - 2 < after) after = total - g - 2 > 0 ? total - g - 2 : 0;
    wait_slabs_le<D>(after);
    __syncthreads();
    {
      const bool ld = !TAIL || g + NS < total;
      const bool ldw = !TAIL || (ld && d_whole());
      const uint32_t la = la_of(d_g), lb = lb_of(d_g);
      if (TAIL && ld && !ldw) dma_tail(la, lb, 0, DH);
      kstep(Y, X, st_base(g + 1), 0, ldw, la, lb, 0);
    }
  };

  // ---- prologue: slabs 0 .. NS-2 and the first half of slab NS-1 in
  // flight, slab 0 visible, K-step 0 of slab 0 in X.
  const int nfull = !TAIL || total >= NS - 1 ? NS - 1 : total;
  for (int i = 0; i < nfull; ++i) {
    dma_range(0, D);
    dma_advance();
  }
  const bool half = !TAIL || NS - 1 < total;
  if (half) dma_range(0, DH);
  wait_loads_le<D, DH>((nfull - 1) * D + (half ? DH : 0));
  __syncthreads();
#pragma unroll
  for (int r = 0; r < NREAD; ++r) read_one(X, st_base(0), 0, r);

  constexpr int CPR = S::WN / 8;                 // 16-byte chunks per staged row
  constexpr int ROWB = S::ROWB;
  char* const cst = smem + NS * S::STAGE + wave * (32 * ROWB);

  int g = 0;
  unsigned int taken = ~0u;
  int unpublished = 0;   // first of this workgroup's blocks whose tiles are not yet published
  for (int lb = 0; lb < mine; ++lb) {
    const BlockPos bp = block_of_position(a.order, w + lb * G, grid);
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
      for (int j = 0; j < S::FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
    for (int kt = 0; kt < nk; ++kt) step(g++);

    // Taken by thread 0 and made wave-uniform, so it waits in a scalar
    // register (meaningful in wave 0 only).
    if (a.take_ctr && wave == 0 && lb + 1 == mine) {
      const unsigned int t = tid == 0 ? atomicAdd(a.take_ctr, 1u) : 0u;
      taken = __builtin_amdgcn_readfirstlane(t);
    }

    // ---- epilogue.  Lane holds D[n][m] for m = lane % 32 and
    // n = 8 (v / 4) + 4 (lane / 32) + v % 4, v = 0..15 (D = C^T): 4
    // consecutive columns of one row per group of 4 registers.  32 rows at a
    // time are staged in this wave's own LDS area (16-byte chunks
    // XOR-swizzled by row), then stored as whole rows with 16-byte lanes, so
    // every store instruction writes full 128-byte lines.
    // The store mode is chosen once per block, so the unrolled stores carry
    // no per-store branch.
    uint16_t* cblk = a.C + static_cast<int64_t>(bp.mb * BM + wm * S::WM) * a.ldc + bp.nb * BN + wn * S::WN;
    auto epilogue = [&](auto mode) {
      constexpr int SM = decltype(mode)::value;
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
      // Lanes read rows other lanes wrote: synchronise the wave (lanes are
      // separate threads to the compiler, which may otherwise move the reads).
      wave_sync();
      constexpr int RPI = 64 / CPR;              // rows per store instruction
#pragma unroll
      for (int r0 = 0; r0 < 32; r0 += RPI) {
        const int rr = r0 + lane / CPR, c = lane % CPR;
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(cst + rr * ROWB + ((c ^ (rr % CPR)) << 4));
        uint16_t* dst = cblk + static_cast<int64_t>(i * 32 + rr) * a.ldc + c * 8;
        if (SM == 1) __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t*>(dst));
        else if (SM == 2) *reinterpret_cast<u32x4_t*>(dst) = v;
        else store16_wt(dst, v);
      }
      wave_sync();                               // the next round rewrites these rows
    }
    };
    if (a.store_mode == 1) epilogue(IC<1>{});
    else if (a.store_mode == 2) epilogue(IC<2>{});
    else epilogue(IC<0>{});

    // Release granularity (paper Section 5.3.2): one release covers the
    // tiles of every block since the last publication.  With release groups
    // every block is released into its group's counter, and the workgroup
    // whose block completes the group publishes the group's flags.
    //
    // A release starts with every wave waiting for its own tile stores: they
    // are inline asm, hidden from the compiler's wait tracking, so neither
    // the barrier nor a fence in another wave waits for them.  Write-through
    // stores are then in memory, where every XCD's acquire finds them, and
    // the flags can follow at once; non-temporal stores may still sit dirty
    // in this XCD's L2 and need the fence's write-back first.
    const bool grouped = a.release_blocks <= kReleasePartition;
    const bool release = a.flags != nullptr && (grouped || lb + 1 == mine ||
                                                (a.release_blocks >= 1 && lb + 1 - unpublished >= a.release_blocks));
    if (release && grouped) {
      const int tiles_n = a.N / kTile;
      const int part_rows = a.M / a.P;
      const int d = a.release_blocks == kReleasePartition ? bp.mb * BM / part_rows : 0;
      const int64_t first = a.release_blocks == kReleasePartition ? static_cast<int64_t>(d) * (part_rows / kTile) * tiles_n : 0;
      const int64_t count = static_cast<int64_t>(a.release_blocks == kReleasePartition ? part_rows : a.M) / kTile * tiles_n;
      int* const s_last = reinterpret_cast<int*>(smem + NS * S::STAGE);   // wave 0's staging rows, free here
      wait_vm<0>();
      __syncthreads();
      if (tid == 0) {
        if (a.store_mode != 0) release_fence();
        constexpr unsigned long long c = (BM / kTile) * (BN / kTile);
        unsigned long long* ctr = a.group_ctr + (a.release_blocks == kReleasePartition ? d : a.P);
        const unsigned long long old = atomicAdd(ctr, c);
        // every block of the group was released before it was counted
        *s_last = (old + c) % static_cast<unsigned long long>(count) == 0;
      }
      __syncthreads();
      if (*s_last)
        for (int64_t i = tid; i < count; i += 256) publish_relaxed(a.flags + first + i, a.epoch);
      __syncthreads();   // s_last lives in staging rows the next epilogue rewrites
      unpublished = lb + 1;
    } else if (release) {
      wait_vm<0>();
      __syncthreads();
      if (tid == 0) {
        const int tiles_n = a.N / kTile;
        if (a.store_mode != 0) release_fence();
        for (int pb = unpublished; pb <= lb; ++pb) {
          const BlockPos pp = pb == lb ? bp : block_of_position(a.order, w + pb * G, grid);
#pragma unroll
          for (int ti = 0; ti < BM / kTile; ++ti)
#pragma unroll
            for (int tj = 0; tj < BN / kTile; ++tj)
              publish_relaxed(a.flags + (pp.mb * (BM / kTile) + ti) * tiles_n + pp.nb * (BN / kTile) + tj,
                              a.epoch);
        }
      }
      unpublished = lb + 1;
    }
  }
  // Loads past the end of the stream may still be writing LDS.
  if (!TAIL) wait_vm<0>();
  return taken;
}

template <int BM, int BN, bool TAIL>
__global__ __launch_bounds__(256) void gemm_producer(GemmArgs a) {
  __shared__ __attribute__((aligned(1024))) char smem[GemmShape<BM, BN>::LDS_BYTES];
  producer_body<BM, BN, TAIL>(a, blockIdx.x, gridDim.x, smem);
}

}  // namespace entwine
