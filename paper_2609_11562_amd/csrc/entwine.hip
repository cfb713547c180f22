// entwine.hip - host launcher and C ABI of libentwine.so (declared in
// include/entwine.h).
//
// One call of the fused path (paper Section 4.1): fork the reduce stream off
// the GEMM stream, enqueue the producer GEMM on the GEMM stream and, on the
// reduce stream, the synthetic peer-flag publication followed by the tile
// reducer, then join the reduce stream back into the GEMM stream.  The GEMM
// is enqueued first, so it can never be starved by waiting reducer
// workgroups: if both streams land on one hardware queue the reducer simply
// runs after the GEMM.  Flags are never cleared between calls; every call
// takes a fresh epoch and a flag is ready when it holds that epoch (the
// paper resets flags before each invocation).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/entwine.h"
#include "gemm_producer.h"
#include "gemm_reduce_fused.h"
#include "tile_order.h"
#include "tile_reducer.h"

using namespace entwine;

namespace {

constexpr int kRing = 256;
constexpr int kStampWgs = 1024;   // workgroups with per-call timestamps (single launch)

struct TimingSlot {
  hipEvent_t start = nullptr, gemm_end = nullptr, red_end = nullptr;
  bool has_gemm = false, has_red = false;
  bool has_stamps = false;   // single launch: role spans from device timestamps
  int G = 0, grid = 0;
};

struct CfgShape {
  int BM, BN;
};
constexpr CfgShape kCfgShapes[ENTWINE_GEMM_NUM_CFGS] = {{256, 256}, {256, 128}, {128, 256}, {128, 128}};

}  // namespace

struct entwine_ctx {
  int device = 0;
  int64_t M = 0, N = 0, K = 0;
  int P = 1;
  int cus = 0;
  int64_t ntiles = 0;
  int* flags = nullptr;        // local tile flags
  int* peer_flags = nullptr;   // (P-1) x ntiles
  int* status = nullptr;       // {code, tile, src, pad}
  uint16_t* scratch = nullptr; // M x N partial when the caller passes none
  uint16_t* zeros = nullptr;   // zero page read by the producer for the K tail
  uint32_t epoch = 0;
  uint64_t ticks_per_us = 100;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  TimingSlot ring[kRing];
  unsigned long long* stamps = nullptr;   // kRing x kStampWgs x kStampsPerWg, on first need
  unsigned int* task_ctr = nullptr;       // single launch: {next task, finished workgroups}, zero between calls
  unsigned long long* group_ctr = nullptr;  // release groups: tiles stored per partition (P) and output (1)
  int64_t ncalls = 0;          // calls with record_timing
  hipStream_t last_stream = nullptr;
  std::string err;
};

namespace {

thread_local std::string g_err;

entwine_status fail(entwine_ctx* ctx, entwine_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (ctx) ctx->err = buf;
  g_err = buf;
  return s;
}

#define HIP_OR_FAIL(ctx, call)                                                           \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess) return fail(ctx, ENTWINE_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

entwine_status validate_shape(entwine_ctx* ctx, int64_t M, int64_t N, int64_t K, int32_t P) {
  if (P < 1 || P > ENTWINE_MAX_P) return fail(ctx, ENTWINE_EINVAL, "P=%d outside [1, %d]", P, ENTWINE_MAX_P);
  if (M <= 0 || N <= 0 || K <= 0) return fail(ctx, ENTWINE_EINVAL, "M, N, K must be positive");
  if (M % (int64_t(ENTWINE_TILE) * P)) return fail(ctx, ENTWINE_EINVAL, "M=%lld is not a multiple of 128*P", (long long)M);
  if (N % ENTWINE_TILE) return fail(ctx, ENTWINE_EINVAL, "N=%lld is not a multiple of 128", (long long)N);
  if (K % 8) return fail(ctx, ENTWINE_EINVAL, "K=%lld is not a multiple of 8", (long long)K);
  if (M > (1 << 30) || N > (1 << 30) || K > (1 << 30)) return fail(ctx, ENTWINE_EINVAL, "dimension too large");
  return ENTWINE_OK;
}

int default_gemm_cfg(int64_t M, int64_t N, int P) {
  for (int c = 0; c < ENTWINE_GEMM_NUM_CFGS; ++c)
    if ((M / P) % kCfgShapes[c].BM == 0 && N % kCfgShapes[c].BN == 0) return c;
  return ENTWINE_GEMM_128x128;
}

struct Resolved {
  // x: dedicated reducer workgroups of the fused launch (0 with reduce_wgs
  // -1); x_alone: grid of the standalone reducer kernel (reduce_only, the
  // sequential form and the two-stream forms), never 0.
  int order, gemm_cfg, BM, BN, x, x_alone, threads, withhold, timing, group_m, gemm_wgs, launch, release_blocks,
      store_mode;
  uint64_t timeout_us;
};

entwine_status resolve(entwine_ctx* ctx, int64_t M, int64_t N, int32_t P, int32_t dest,
                       const entwine_config* cfg, int cus, Resolved* r) {
  entwine_config c;
  entwine_config_default(&c);
  if (cfg) c = *cfg;
  if (dest != ENTWINE_DEST_ALL && (dest < 0 || dest >= P))
    return fail(ctx, ENTWINE_EINVAL, "dest=%d outside [-1, P)", dest);
  if (c.order < 0 || c.order > 2) return fail(ctx, ENTWINE_EINVAL, "unknown order %d", c.order);
  if (c.gemm_cfg < -1 || c.gemm_cfg >= ENTWINE_GEMM_NUM_CFGS) return fail(ctx, ENTWINE_EINVAL, "unknown gemm_cfg %d", c.gemm_cfg);
  if (c.reduce_threads != 0 && c.reduce_threads != 128 && c.reduce_threads != 256 && c.reduce_threads != 512 &&
      c.reduce_threads != 1024)
    return fail(ctx, ENTWINE_EINVAL, "reduce_threads must be 128, 256, 512 or 1024");
  if (c.reduce_wgs < -1 || (c.reduce_wgs == -1 && c.launch != 0))
    return fail(ctx, ENTWINE_EINVAL, "reduce_wgs must be >= 0 (or -1 with launch 0)");
  if (c.timeout_us < 0) return fail(ctx, ENTWINE_EINVAL, "timeout_us must be >= 0");
  if (c.withhold_peer < -1 || c.withhold_peer > P - 2) return fail(ctx, ENTWINE_EINVAL, "withhold_peer outside [-1, P-2]");
  if (c.group_m < 0 || c.group_m > 64) return fail(ctx, ENTWINE_EINVAL, "group_m outside [0, 64]");
  if (c.gemm_wgs < 0) return fail(ctx, ENTWINE_EINVAL, "gemm_wgs must be >= 0");
  if (c.launch < 0 || c.launch > 2) return fail(ctx, ENTWINE_EINVAL, "launch must be 0, 1 or 2");
  if (c.release_blocks < -3) return fail(ctx, ENTWINE_EINVAL, "release_blocks must be >= -3");
  if (c.store_mode < 0 || c.store_mode > 2) return fail(ctx, ENTWINE_EINVAL, "store_mode must be 0, 1 or 2");
  r->order = c.order;
  r->gemm_cfg = c.gemm_cfg < 0 ? default_gemm_cfg(M, N, P) : c.gemm_cfg;
  r->BM = kCfgShapes[r->gemm_cfg].BM;
  r->BN = kCfgShapes[r->gemm_cfg].BN;
  if ((M / P) % r->BM || N % r->BN)
    return fail(ctx, ENTWINE_EUNSUPPORTED, "block %dx%d does not divide the %lldx%lld chunk", r->BM, r->BN,
                (long long)(M / P), (long long)N);
  const int Q = tiles_per_partition(int(M), int(N), P);
  // Default budget: 16 dedicated reducer CUs; in the shared pool one reducer
  // workgroup per CU.
  int x = c.reduce_wgs > 0 ? c.reduce_wgs : (c.launch == 2 ? std::max(16, cus) : 16);
  const int cap_cus = std::max(1, (cus > 1 ? cus - 1 : 255));
  if (dest == ENTWINE_DEST_ALL) {
    x = std::min(x, Q * P);
    x = ((x + P - 1) / P) * P;
    while (x > P && x > cap_cus) x -= P;
  } else {
    x = std::min(std::min(x, Q), cap_cus);
  }
  r->x_alone = std::max(x, 1);
  // The single launch defaults to no dedicated reducers: producers reduce
  // once their blocks are done, which measured fastest on most shapes.
  r->x = c.reduce_wgs == -1 || (c.reduce_wgs == 0 && c.launch == 0) ? 0 : r->x_alone;
  r->threads = c.reduce_threads ? c.reduce_threads : 1024;
  r->withhold = c.withhold_peer;
  r->timing = c.record_timing;
  r->timeout_us = c.timeout_us ? uint64_t(c.timeout_us) : 2000000ull;
  r->group_m = c.group_m ? c.group_m : 4;
  r->gemm_wgs = c.gemm_wgs;
  r->launch = c.launch;
  r->release_blocks = c.release_blocks == 0 ? 2 : c.release_blocks;   // -1: at the end; -2, -3: groups
  r->store_mode = c.store_mode;
  return ENTWINE_OK;
}

entwine_status check_matrix(entwine_ctx* ctx, const void* p, int64_t ld, int64_t cols, const char* name) {
  if (!p) return fail(ctx, ENTWINE_EINVAL, "%s is NULL", name);
  if (!aligned16(p)) return fail(ctx, ENTWINE_EINVAL, "%s is not 16-byte aligned", name);
  if (ld < cols) return fail(ctx, ENTWINE_EINVAL, "ld of %s (%lld) < %lld", name, (long long)ld, (long long)cols);
  if (ld % 8) return fail(ctx, ENTWINE_EINVAL, "ld of %s is not a multiple of 8", name);
  return ENTWINE_OK;
}

#define CHECK(x)                       \
  do {                                 \
    entwine_status s_ = (x);           \
    if (s_ != ENTWINE_OK) return s_;   \
  } while (0)

typedef void (*GemmKernel)(GemmArgs);
template <bool TAIL>
GemmKernel gemm_kernel_t(int cfg) {
  switch (cfg) {
    case 0: return gemm_producer<256, 256, TAIL>;
    case 1: return gemm_producer<256, 128, TAIL>;
    case 2: return gemm_producer<128, 256, TAIL>;
    default: return gemm_producer<128, 128, TAIL>;
  }
}
// The tail variant handles K % 32 != 0 (slab width of the producer).
GemmKernel gemm_kernel(int cfg, int64_t K) {
  return K % GemmShape<128, 128>::BK ? gemm_kernel_t<true>(cfg) : gemm_kernel_t<false>(cfg);
}

typedef void (*ReduceKernel)(ReduceArgs);
template <int T>
ReduceKernel reduce_kernel_p(int P) {
  switch (P) {
    case 1: return tile_reducer<T, 1>;
    case 2: return tile_reducer<T, 2>;
    case 3: return tile_reducer<T, 3>;
    case 4: return tile_reducer<T, 4>;
    case 5: return tile_reducer<T, 5>;
    case 6: return tile_reducer<T, 6>;
    case 7: return tile_reducer<T, 7>;
    default: return tile_reducer<T, 8>;
  }
}
ReduceKernel shared_reduce_kernel(int P) {
  switch (P) {
    case 1: return tile_reducer_shared<1>;
    case 2: return tile_reducer_shared<2>;
    case 3: return tile_reducer_shared<3>;
    case 4: return tile_reducer_shared<4>;
    case 5: return tile_reducer_shared<5>;
    case 6: return tile_reducer_shared<6>;
    case 7: return tile_reducer_shared<7>;
    default: return tile_reducer_shared<8>;
  }
}

ReduceKernel reduce_kernel(int threads, int P) {
  if (threads == 128) return reduce_kernel_p<128>(P);
  if (threads == 512) return reduce_kernel_p<512>(P);
  if (threads == 1024) return reduce_kernel_p<1024>(P);
  return reduce_kernel_p<256>(P);
}

uint32_t next_epoch(entwine_ctx* ctx) {
  ctx->epoch += 1;
  if (ctx->epoch == 0 || ctx->epoch > 0x7fffffffu) ctx->epoch = 1;  // flags compare as int
  return ctx->epoch;
}

entwine_status ensure_scratch(entwine_ctx* ctx) {
  if (ctx->scratch) return ENTWINE_OK;
  hipError_t e = hipMalloc(&ctx->scratch, size_t(ctx->M) * size_t(ctx->N) * 2);
  if (e != hipSuccess) {
    ctx->scratch = nullptr;
    return fail(ctx, ENTWINE_ENOMEM, "partial scratch: %s", hipGetErrorString(e));
  }
  return ENTWINE_OK;
}

TimingSlot* timing_slot(entwine_ctx* ctx, const Resolved& r) {
  if (!r.timing) return nullptr;
  TimingSlot* s = &ctx->ring[ctx->ncalls % kRing];
  ctx->ncalls++;
  s->has_gemm = s->has_red = s->has_stamps = false;
  return s;
}

// Producer grid: persistent workgroups, one per CU, each walking positions
// w, w + G, ...  G is a multiple of 8 so that position p keeps running on XCD
// p mod 8 (workgroups are dispatched round-robin over the 8 XCDs).  In the
// fused path the reducer's x workgroups get the remaining CUs.
int producer_grid(const entwine_ctx* ctx, const Resolved& r, bool fused) {
  const int nblk = int((ctx->M / r.BM) * (ctx->N / r.BN));
  const int cus = ctx->cus > 0 ? ctx->cus : 256;
  int g = r.gemm_wgs;
  if (g <= 0) {
    g = fused ? cus - r.x : cus;
    g = std::max(8, (g / 8) * 8);
  }
  // One launch holding both roles: keep every workgroup resident.
  if (fused && r.launch == 0) g = std::max(1, std::min(g, cus - r.x));
  return std::min(g, nblk);
}

GemmArgs gemm_args(entwine_ctx* ctx, const Resolved& r, const void* A, int64_t lda, const void* B, int64_t ldb,
                   void* C, int64_t ldc, bool publish, uint32_t epoch) {
  GemmArgs g;
  g.A = static_cast<const uint16_t*>(A);
  g.B = static_cast<const uint16_t*>(B);
  g.C = static_cast<uint16_t*>(C);
  g.zeros = ctx->zeros;
  g.lda = lda;
  g.ldb = ldb;
  g.ldc = ldc;
  g.M = int(ctx->M);
  g.N = int(ctx->N);
  g.K = int(ctx->K);
  g.P = ctx->P;
  g.order = r.order;
  g.group_m = r.group_m;
  g.flags = publish ? ctx->flags : nullptr;
  g.epoch = epoch;
  g.release_blocks = r.release_blocks;
  g.store_mode = r.store_mode;
  g.group_ctr = ctx->group_ctr;
  g.take_ctr = nullptr;
  return g;
}

entwine_status launch_gemm(entwine_ctx* ctx, const Resolved& r, const void* A, int64_t lda, const void* B,
                           int64_t ldb, void* C, int64_t ldc, bool publish, uint32_t epoch,
                           hipStream_t s, bool fused) {
  const GemmArgs g = gemm_args(ctx, r, A, lda, B, ldb, C, ldc, publish, epoch);
  hipLaunchKernelGGL(gemm_kernel(r.gemm_cfg, ctx->K), dim3(producer_grid(ctx, r, fused)), dim3(256), 0, s, g);
  HIP_OR_FAIL(ctx, hipGetLastError());
  return ENTWINE_OK;
}

entwine_status launch_publish(entwine_ctx* ctx, int* flags, int64_t n, int64_t per, int skip, uint32_t epoch,
                              hipStream_t s) {
  if (n <= 0) return ENTWINE_OK;
  const int blocks = int(std::min<int64_t>((n + 255) / 256, 1024));
  hipLaunchKernelGGL(publish_fill, dim3(blocks), dim3(256), 0, s, flags, n, per, skip, epoch);
  HIP_OR_FAIL(ctx, hipGetLastError());
  return ENTWINE_OK;
}

ReduceArgs reduce_args(entwine_ctx* ctx, const Resolved& r, const void* partial, int64_t ldc,
                       const void* const* peers, int64_t ldp, int32_t dest, void* out, int64_t ldo,
                       uint32_t epoch) {
  ReduceArgs ra;
  memset(&ra, 0, sizeof ra);
  ra.partial = static_cast<const uint16_t*>(partial);
  for (int q = 0; q < ctx->P - 1; ++q) ra.peers[q] = static_cast<const uint16_t*>(peers[q]);
  ra.out = static_cast<uint16_t*>(out);
  ra.ldc = ldc;
  ra.ldp = ldp;
  ra.ldo = ldo;
  ra.M = int(ctx->M);
  ra.N = int(ctx->N);
  ra.dest = dest;
  ra.x = r.x_alone;
  ra.BM = r.BM;
  ra.BN = r.BN;
  ra.group_m = r.group_m;
  ra.flags = ctx->flags;
  ra.peer_flags = ctx->peer_flags;
  ra.epoch = epoch;
  ra.status = ctx->status;
  ra.timeout_ticks = r.timeout_us * ctx->ticks_per_us;
  ra.publish_peers = 0;
  ra.withhold_peer = r.withhold;
  return ra;
}

entwine_status launch_reduce(entwine_ctx* ctx, const Resolved& r, const void* partial, int64_t ldc,
                             const void* const* peers, int64_t ldp, int32_t dest, void* out, int64_t ldo,
                             uint32_t epoch, hipStream_t s) {
  const ReduceArgs ra = reduce_args(ctx, r, partial, ldc, peers, ldp, dest, out, ldo, epoch);
  hipLaunchKernelGGL(reduce_kernel(r.threads, ctx->P), dim3(r.x_alone), dim3(r.threads), 0, s, ra);
  HIP_OR_FAIL(ctx, hipGetLastError());
  return ENTWINE_OK;
}

// Shared pool: reducers of 256 threads beside the producers on the same CUs,
// publishing the synthetic peers' flags themselves.
entwine_status launch_reduce_shared(entwine_ctx* ctx, const Resolved& r, const void* partial, int64_t ldc,
                                    const void* const* peers, int64_t ldp, int32_t dest, void* out, int64_t ldo,
                                    uint32_t epoch, hipStream_t s) {
  // The shared-pool reducer addresses every matrix with 32-bit byte offsets.
  const int64_t rows = ctx->M;
  for (int64_t ld : {ldc, ldp, ldo})
    if ((rows * ld + ctx->N) * 2 > (int64_t(1) << 32))
      return fail(ctx, ENTWINE_EUNSUPPORTED, "launch=2 needs matrices under 4 GiB (ld %lld)", (long long)ld);
  ReduceArgs ra = reduce_args(ctx, r, partial, ldc, peers, ldp, dest, out, ldo, epoch);
  ra.publish_peers = 1;
  hipLaunchKernelGGL(shared_reduce_kernel(ctx->P), dim3(r.x_alone), dim3(256), 0, s, ra);
  HIP_OR_FAIL(ctx, hipGetLastError());
  return ENTWINE_OK;
}

typedef void (*FusedKernel)(GemmArgs, ReduceArgs, int, int, unsigned long long*);
template <bool TAIL>
FusedKernel fused_kernel_t(int cfg) {
  switch (cfg) {
    case 0: return gemm_reduce_fused<256, 256, TAIL>;
    case 1: return gemm_reduce_fused<256, 128, TAIL>;
    case 2: return gemm_reduce_fused<128, 256, TAIL>;
    default: return gemm_reduce_fused<128, 128, TAIL>;
  }
}

// The fused path as one launch on stream s: G producer workgroups, then x
// reducers of 256 threads that also publish the synthetic peers' flags.
struct LayerArgs {
  const void* residual;
  int64_t ldr;
  const void* gamma;
  float eps;
  void* y;
  int64_t ldy;
};

entwine_status launch_fused(entwine_ctx* ctx, const Resolved& r, const GemmArgs& g, const void* partial,
                            int64_t ldc, const void* const* peers, int64_t ldp, int32_t dest, void* out,
                            int64_t ldo, uint32_t epoch, TimingSlot* ts, hipStream_t s,
                            const LayerArgs* layer = nullptr) {
  ReduceArgs ra = reduce_args(ctx, r, partial, ldc, peers, ldp, dest, out, ldo, epoch);
  ra.task_ctr = ctx->task_ctr;
  ra.call_tiles = tiles_per_partition(int(ctx->M), int(ctx->N), ctx->P) * (dest == ENTWINE_DEST_ALL ? ctx->P : 1);
  ra.ntasks = kTaskSplit * ra.call_tiles;   // reducer_dynamic
  if (layer) {
    // One task per output row (reducer_layer).
    ra.layer = 1;
    ra.ntasks = int(dest == ENTWINE_DEST_ALL ? ctx->M : ctx->M / ctx->P);
    ra.residual = static_cast<const uint16_t*>(layer->residual);
    ra.ldr = layer->ldr;
    ra.gamma = static_cast<const uint16_t*>(layer->gamma);
    ra.eps = layer->eps;
    ra.y = static_cast<uint16_t*>(layer->y);
    ra.ldy = layer->ldy;
  }
  const int G = producer_grid(ctx, r, true);
  const int grid = G + r.x;
  unsigned long long* stamps = nullptr;
  if (ts && grid <= kStampWgs) {
    if (!ctx->stamps)
      HIP_OR_FAIL(ctx, hipMalloc(&ctx->stamps, size_t(kRing) * kStampWgs * kStampsPerWg * sizeof(unsigned long long)));
    stamps = ctx->stamps + size_t(ts - ctx->ring) * kStampWgs * kStampsPerWg;
    ts->has_stamps = true;
    ts->G = G;
    ts->grid = grid;
  }
  FusedKernel k = ctx->K % GemmShape<128, 128>::BK ? fused_kernel_t<true>(r.gemm_cfg) : fused_kernel_t<false>(r.gemm_cfg);
  GemmArgs gf = g;
  gf.take_ctr = ctx->task_ctr;   // producers take their first reduction task early
  hipLaunchKernelGGL(k, dim3(grid), dim3(256), 0, s, gf, ra, G, ctx->P, stamps);
  HIP_OR_FAIL(ctx, hipGetLastError());
  return ENTWINE_OK;
}

// The producer addresses A and B with 32-bit byte offsets inside a block.
entwine_status check_operand_ld(entwine_ctx* ctx, int64_t lda, int64_t ldb) {
  if (lda > (int64_t(1) << 22) || ldb > (int64_t(1) << 22))
    return fail(ctx, ENTWINE_EINVAL, "lda/ldb above 2^22 elements are not supported");
  return ENTWINE_OK;
}

entwine_status check_peers(entwine_ctx* ctx, const void* const* peers, int64_t ldp) {
  if (ctx->P == 1) return ENTWINE_OK;
  if (!peers) return fail(ctx, ENTWINE_EINVAL, "peers is NULL with P > 1");
  for (int q = 0; q < ctx->P - 1; ++q) CHECK(check_matrix(ctx, peers[q], ldp, ctx->N, "peer"));
  return ENTWINE_OK;
}

}  // namespace

extern "C" {

void entwine_config_default(entwine_config* cfg) {
  if (!cfg) return;
  cfg->order = ENTWINE_ORDER_INTERLEAVED;
  cfg->gemm_cfg = -1;
  cfg->reduce_wgs = 0;
  cfg->reduce_threads = 0;
  cfg->timeout_us = 0;
  cfg->withhold_peer = -1;
  cfg->record_timing = 0;
  cfg->group_m = 0;
  cfg->gemm_wgs = 0;
  cfg->launch = 0;
  cfg->release_blocks = 0;
  cfg->store_mode = 0;
}

int32_t entwine_abi_version(void) { return ENTWINE_ABI_VERSION; }

const char* entwine_status_string(entwine_status s) {
  switch (s) {
    case ENTWINE_OK: return "ENTWINE_OK";
    case ENTWINE_EINVAL: return "ENTWINE_EINVAL";
    case ENTWINE_EUNSUPPORTED: return "ENTWINE_EUNSUPPORTED";
    case ENTWINE_ENOMEM: return "ENTWINE_ENOMEM";
    case ENTWINE_EHIP: return "ENTWINE_EHIP";
    case ENTWINE_ETIMEOUT: return "ENTWINE_ETIMEOUT";
  }
  return "ENTWINE_UNKNOWN";
}

const char* entwine_last_error(const entwine_ctx* ctx) { return ctx ? ctx->err.c_str() : g_err.c_str(); }

entwine_status entwine_validate(int64_t M, int64_t N, int64_t K, int32_t P, int32_t dest,
                                const entwine_config* cfg) {
  CHECK(validate_shape(nullptr, M, N, K, P));
  Resolved r;
  return resolve(nullptr, M, N, P, dest, cfg, 256, &r);
}

entwine_status entwine_ctx_create(entwine_ctx** out, int32_t device, int64_t M, int64_t N, int64_t K,
                                  int32_t P) {
  if (!out) return fail(nullptr, ENTWINE_EINVAL, "out is NULL");
  *out = nullptr;
  CHECK(validate_shape(nullptr, M, N, K, P));
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
    return fail(nullptr, ENTWINE_EINVAL, "device %d not available", device);
  entwine_ctx* c = new entwine_ctx();
  c->device = device;
  c->M = M;
  c->N = N;
  c->K = K;
  c->P = P;
  c->ntiles = (M / ENTWINE_TILE) * (N / ENTWINE_TILE);
  auto bail = [&](entwine_status s) {
    entwine_ctx_destroy(c);
    return s;
  };
  if (hipSetDevice(device) != hipSuccess) return bail(fail(nullptr, ENTWINE_EHIP, "hipSetDevice failed"));
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, device) != hipSuccess) return bail(fail(nullptr, ENTWINE_EHIP, "device properties"));
  c->cus = prop.multiProcessorCount;
  int khz = 0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, device) == hipSuccess && khz > 0)
    c->ticks_per_us = uint64_t(khz) / 1000 ? uint64_t(khz) / 1000 : 1;
  const size_t fbytes = size_t(c->ntiles) * sizeof(int);
  if (hipMalloc(&c->flags, fbytes) != hipSuccess ||
      hipMalloc(&c->peer_flags, fbytes * size_t(P > 1 ? P - 1 : 1)) != hipSuccess ||
      hipMalloc(&c->status, 4 * sizeof(int)) != hipSuccess || hipMalloc(&c->zeros, 256) != hipSuccess ||
      hipMalloc(&c->task_ctr, 2 * sizeof(unsigned int)) != hipSuccess ||
      hipMalloc(&c->group_ctr, size_t(P + 1) * sizeof(unsigned long long)) != hipSuccess)
    return bail(fail(nullptr, ENTWINE_ENOMEM, "flag allocation failed"));
  if (hipMemset(c->flags, 0, fbytes) != hipSuccess ||
      hipMemset(c->peer_flags, 0, fbytes * size_t(P > 1 ? P - 1 : 1)) != hipSuccess ||
      hipMemset(c->status, 0, 4 * sizeof(int)) != hipSuccess || hipMemset(c->zeros, 0, 256) != hipSuccess ||
      hipMemset(c->task_ctr, 0, 2 * sizeof(unsigned int)) != hipSuccess ||
      hipMemset(c->group_ctr, 0, size_t(P + 1) * sizeof(unsigned long long)) != hipSuccess)
    return bail(fail(nullptr, ENTWINE_EHIP, "flag initialisation failed"));
  if (hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming) != hipSuccess)
    return bail(fail(nullptr, ENTWINE_EHIP, "event creation failed"));
  for (auto& s : c->ring)
    if (hipEventCreate(&s.start) != hipSuccess || hipEventCreate(&s.gemm_end) != hipSuccess ||
        hipEventCreate(&s.red_end) != hipSuccess)
      return bail(fail(nullptr, ENTWINE_EHIP, "event creation failed"));
  if (hipDeviceSynchronize() != hipSuccess) return bail(fail(nullptr, ENTWINE_EHIP, "initial sync failed"));
  *out = c;
  return ENTWINE_OK;
}

entwine_status entwine_ctx_destroy(entwine_ctx* ctx) {
  if (!ctx) return ENTWINE_OK;
  (void)hipSetDevice(ctx->device);
  (void)hipDeviceSynchronize();
  if (ctx->flags) (void)hipFree(ctx->flags);
  if (ctx->peer_flags) (void)hipFree(ctx->peer_flags);
  if (ctx->status) (void)hipFree(ctx->status);
  if (ctx->scratch) (void)hipFree(ctx->scratch);
  if (ctx->zeros) (void)hipFree(ctx->zeros);
  if (ctx->stamps) (void)hipFree(ctx->stamps);
  if (ctx->task_ctr) (void)hipFree(ctx->task_ctr);
  if (ctx->group_ctr) (void)hipFree(ctx->group_ctr);
  if (ctx->ev_fork) (void)hipEventDestroy(ctx->ev_fork);
  if (ctx->ev_join) (void)hipEventDestroy(ctx->ev_join);
  for (auto& s : ctx->ring) {
    if (s.start) (void)hipEventDestroy(s.start);
    if (s.gemm_end) (void)hipEventDestroy(s.gemm_end);
    if (s.red_end) (void)hipEventDestroy(s.red_end);
  }
  delete ctx;
  return ENTWINE_OK;
}

entwine_status entwine_gemm_rs(entwine_ctx* ctx, const void* A, int64_t lda, const void* B, int64_t ldb,
                               const void* const* peers, int64_t ldp, int32_t dest, void* out, int64_t ldo,
                               void* partial, int64_t ldc, const entwine_config* cfg, void* gemm_stream,
                               void* reduce_stream) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  Resolved r;
  CHECK(resolve(ctx, ctx->M, ctx->N, ctx->P, dest, cfg, ctx->cus, &r));
  CHECK(check_matrix(ctx, A, lda, ctx->K, "A"));
  CHECK(check_matrix(ctx, B, ldb, ctx->N, "B"));
  CHECK(check_operand_ld(ctx, lda, ldb));
  CHECK(check_matrix(ctx, out, ldo, ctx->N, "out"));
  CHECK(check_peers(ctx, peers, ldp));
  if (partial) {
    CHECK(check_matrix(ctx, partial, ldc, ctx->N, "partial"));
  } else {
    CHECK(ensure_scratch(ctx));
    partial = ctx->scratch;
    ldc = ctx->N;
  }
  HIP_OR_FAIL(ctx, hipSetDevice(ctx->device));
  hipStream_t gs = static_cast<hipStream_t>(gemm_stream);
  hipStream_t rs = static_cast<hipStream_t>(reduce_stream);
  const bool fused = gs != rs;
  const uint32_t epoch = next_epoch(ctx);
  TimingSlot* ts = timing_slot(ctx, r);

  if (fused && r.launch == 0) {
    if (ts) HIP_OR_FAIL(ctx, hipEventRecord(ts->start, gs));
    const GemmArgs g = gemm_args(ctx, r, A, lda, B, ldb, partial, ldc, true, epoch);
    CHECK(launch_fused(ctx, r, g, partial, ldc, peers, ldp, dest, out, ldo, epoch, ts, gs));
    if (ts) {
      HIP_OR_FAIL(ctx, hipEventRecord(ts->red_end, gs));
      ts->has_red = true;
    }
    ctx->last_stream = gs;
    return ENTWINE_OK;
  }

  const bool shared = fused && r.launch == 2;
  if (fused) HIP_OR_FAIL(ctx, hipEventRecord(ctx->ev_fork, gs));
  if (ts) HIP_OR_FAIL(ctx, hipEventRecord(ts->start, gs));
  CHECK(launch_gemm(ctx, r, A, lda, B, ldb, partial, ldc, true, epoch, gs, fused && !shared));
  if (ts) {
    HIP_OR_FAIL(ctx, hipEventRecord(ts->gemm_end, gs));
    ts->has_gemm = true;
  }
  if (fused) HIP_OR_FAIL(ctx, hipStreamWaitEvent(rs, ctx->ev_fork, 0));
  if (shared) {
    CHECK(launch_reduce_shared(ctx, r, partial, ldc, peers, ldp, dest, out, ldo, epoch, rs));
  } else {
    CHECK(launch_publish(ctx, ctx->peer_flags, ctx->ntiles * (ctx->P - 1), ctx->ntiles, r.withhold, epoch, rs));
    CHECK(launch_reduce(ctx, r, partial, ldc, peers, ldp, dest, out, ldo, epoch, rs));
  }
  if (ts) {
    HIP_OR_FAIL(ctx, hipEventRecord(ts->red_end, rs));
    ts->has_red = true;
  }
  if (fused) {
    HIP_OR_FAIL(ctx, hipEventRecord(ctx->ev_join, rs));
    HIP_OR_FAIL(ctx, hipStreamWaitEvent(gs, ctx->ev_join, 0));
  }
  ctx->last_stream = gs;
  return ENTWINE_OK;
}

entwine_status entwine_gemm_rs_rmsnorm(entwine_ctx* ctx, const void* A, int64_t lda, const void* B, int64_t ldb,
                                       const void* const* peers, int64_t ldp, int32_t dest, const void* residual,
                                       int64_t ldr, const void* gamma, float eps, void* h_out, int64_t ldh,
                                       void* y_out, int64_t ldy, void* partial, int64_t ldc,
                                       const entwine_config* cfg, void* stream) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  Resolved r;
  CHECK(resolve(ctx, ctx->M, ctx->N, ctx->P, dest, cfg, ctx->cus, &r));
  if (r.launch != 0) return fail(ctx, ENTWINE_EUNSUPPORTED, "the layer epilogue runs as one launch (launch 0)");
  if (!(eps > 0.0f) || !(eps < 1e30f)) return fail(ctx, ENTWINE_EINVAL, "eps must be positive and finite");
  if (ctx->N > kLayerMaxN) return fail(ctx, ENTWINE_EUNSUPPORTED, "the layer epilogue holds a row in registers: N <= %d", kLayerMaxN);
  CHECK(check_matrix(ctx, A, lda, ctx->K, "A"));
  CHECK(check_matrix(ctx, B, ldb, ctx->N, "B"));
  CHECK(check_operand_ld(ctx, lda, ldb));
  CHECK(check_matrix(ctx, h_out, ldh, ctx->N, "h_out"));
  CHECK(check_matrix(ctx, y_out, ldy, ctx->N, "y_out"));
  CHECK(check_matrix(ctx, residual, ldr, ctx->N, "residual"));
  CHECK(check_matrix(ctx, gamma, ctx->N, ctx->N, "gamma"));
  CHECK(check_peers(ctx, peers, ldp));
  if (partial) {
    CHECK(check_matrix(ctx, partial, ldc, ctx->N, "partial"));
  } else {
    CHECK(ensure_scratch(ctx));
    partial = ctx->scratch;
    ldc = ctx->N;
  }
  HIP_OR_FAIL(ctx, hipSetDevice(ctx->device));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t epoch = next_epoch(ctx);
  TimingSlot* ts = timing_slot(ctx, r);
  if (ts) HIP_OR_FAIL(ctx, hipEventRecord(ts->start, s));
  const GemmArgs g = gemm_args(ctx, r, A, lda, B, ldb, partial, ldc, true, epoch);
  const LayerArgs la{residual, ldr, gamma, eps, y_out, ldy};
  CHECK(launch_fused(ctx, r, g, partial, ldc, peers, ldp, dest, h_out, ldh, epoch, ts, s, &la));
  if (ts) {
    HIP_OR_FAIL(ctx, hipEventRecord(ts->red_end, s));
    ts->has_red = true;
  }
  ctx->last_stream = s;
  return ENTWINE_OK;
}

entwine_status entwine_gemm_only(entwine_ctx* ctx, const void* A, int64_t lda, const void* B, int64_t ldb,
                                 void* partial, int64_t ldc, const entwine_config* cfg, void* stream) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  Resolved r;
  CHECK(resolve(ctx, ctx->M, ctx->N, ctx->P, 0, cfg, ctx->cus, &r));
  CHECK(check_matrix(ctx, A, lda, ctx->K, "A"));
  CHECK(check_matrix(ctx, B, ldb, ctx->N, "B"));
  CHECK(check_operand_ld(ctx, lda, ldb));
  if (partial) {
    CHECK(check_matrix(ctx, partial, ldc, ctx->N, "partial"));
  } else {
    CHECK(ensure_scratch(ctx));
    partial = ctx->scratch;
    ldc = ctx->N;
  }
  HIP_OR_FAIL(ctx, hipSetDevice(ctx->device));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t epoch = next_epoch(ctx);
  TimingSlot* ts = timing_slot(ctx, r);
  if (ts) HIP_OR_FAIL(ctx, hipEventRecord(ts->start, s));
  CHECK(launch_gemm(ctx, r, A, lda, B, ldb, partial, ldc, true, epoch, s, false));
  if (ts) {
    HIP_OR_FAIL(ctx, hipEventRecord(ts->gemm_end, s));
    ts->has_gemm = true;
  }
  ctx->last_stream = s;
  return ENTWINE_OK;
}

entwine_status entwine_reduce_only(entwine_ctx* ctx, const void* partial, int64_t ldc, const void* const* peers,
                                   int64_t ldp, int32_t dest, void* out, int64_t ldo, const entwine_config* cfg,
                                   void* stream) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  Resolved r;
  CHECK(resolve(ctx, ctx->M, ctx->N, ctx->P, dest, cfg, ctx->cus, &r));
  CHECK(check_matrix(ctx, partial, ldc, ctx->N, "partial"));
  CHECK(check_matrix(ctx, out, ldo, ctx->N, "out"));
  CHECK(check_peers(ctx, peers, ldp));
  HIP_OR_FAIL(ctx, hipSetDevice(ctx->device));
  hipStream_t s = static_cast<hipStream_t>(stream);
  const uint32_t epoch = next_epoch(ctx);
  TimingSlot* ts = timing_slot(ctx, r);
  CHECK(launch_publish(ctx, ctx->flags, ctx->ntiles, ctx->ntiles, -1, epoch, s));
  CHECK(launch_publish(ctx, ctx->peer_flags, ctx->ntiles * (ctx->P - 1), ctx->ntiles, r.withhold, epoch, s));
  if (ts) HIP_OR_FAIL(ctx, hipEventRecord(ts->start, s));
  CHECK(launch_reduce(ctx, r, partial, ldc, peers, ldp, dest, out, ldo, epoch, s));
  if (ts) {
    HIP_OR_FAIL(ctx, hipEventRecord(ts->red_end, s));
    ts->has_red = true;
  }
  ctx->last_stream = s;
  return ENTWINE_OK;
}

entwine_status entwine_query_status(entwine_ctx* ctx, int32_t* code, int32_t* tile, int32_t* src) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  HIP_OR_FAIL(ctx, hipSetDevice(ctx->device));
  HIP_OR_FAIL(ctx, hipDeviceSynchronize());
  int h[4] = {0, 0, 0, 0};
  HIP_OR_FAIL(ctx, hipMemcpy(h, ctx->status, sizeof h, hipMemcpyDeviceToHost));
  HIP_OR_FAIL(ctx, hipMemset(ctx->status, 0, sizeof h));
  if (code) *code = h[0];
  if (tile) *tile = h[0] ? h[1] : -1;
  if (src) *src = h[0] ? h[2] : -2;
  if (h[0]) return fail(ctx, ENTWINE_ETIMEOUT, "reducer wait expired on tile %d (source %d)", h[1], h[2]);
  return ENTWINE_OK;
}

// The per-workgroup stamps of a single-launch call, once it has completed.
static entwine_status read_stamps(entwine_ctx* ctx, const TimingSlot& s, std::vector<unsigned long long>& h) {
  HIP_OR_FAIL(ctx, hipEventSynchronize(s.red_end));
  h.resize(size_t(s.grid) * kStampsPerWg);
  HIP_OR_FAIL(ctx, hipMemcpy(h.data(), ctx->stamps + size_t(&s - ctx->ring) * kStampWgs * kStampsPerWg,
                             h.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
  return ENTWINE_OK;
}

entwine_status entwine_last_timing(entwine_ctx* ctx, int32_t back, float* gemm_ms, float* reduce_ms,
                                   float* e2e_ms) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  if (back < 0 || back >= kRing || back >= ctx->ncalls) return fail(ctx, ENTWINE_EINVAL, "no such timed call");
  TimingSlot& s = ctx->ring[(ctx->ncalls - 1 - back) % kRing];
  float g = -1.f, rd = -1.f, e = -1.f;
  if (s.has_stamps) {
    // Single launch: role spans from the workgroups' own timestamps, measured
    // from the first workgroup's start; end to end from the events around it.
    HIP_OR_FAIL(ctx, hipEventSynchronize(s.red_end));
    HIP_OR_FAIL(ctx, hipEventElapsedTime(&e, s.start, s.red_end));
    std::vector<unsigned long long> h;
    CHECK(read_stamps(ctx, s, h));
    unsigned long long t0 = ~0ull, ge = 0, re = 0;
    for (int b = 0; b < s.grid; ++b) {
      t0 = std::min(t0, h[kStampsPerWg * b]);
      if (b < s.G) ge = std::max(ge, h[kStampsPerWg * b + 1]);
      re = std::max(re, h[kStampsPerWg * b + 3]);
    }
    const double per_ms = double(ctx->ticks_per_us) * 1e3;
    g = float(double(ge - t0) / per_ms);
    rd = float(double(re - t0) / per_ms);
    if (gemm_ms) *gemm_ms = g;
    if (reduce_ms) *reduce_ms = rd;
    if (e2e_ms) *e2e_ms = e;
    return ENTWINE_OK;
  }
  if (s.has_gemm) {
    HIP_OR_FAIL(ctx, hipEventSynchronize(s.gemm_end));
    HIP_OR_FAIL(ctx, hipEventElapsedTime(&g, s.start, s.gemm_end));
  }
  if (s.has_red) {
    HIP_OR_FAIL(ctx, hipEventSynchronize(s.red_end));
    HIP_OR_FAIL(ctx, hipEventElapsedTime(&rd, s.start, s.red_end));
  }
  e = std::max(g, rd);
  if (gemm_ms) *gemm_ms = g;
  if (reduce_ms) *reduce_ms = rd;
  if (e2e_ms) *e2e_ms = e;
  return ENTWINE_OK;
}

entwine_status entwine_last_stamps(entwine_ctx* ctx, int32_t back, uint64_t* stamps, int32_t capacity,
                                   int32_t* nwgs, int32_t* nproducers, double* ticks_per_us) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  if (back < 0 || back >= kRing || back >= ctx->ncalls) return fail(ctx, ENTWINE_EINVAL, "no such timed call");
  const TimingSlot& s = ctx->ring[(ctx->ncalls - 1 - back) % kRing];
  if (!s.has_stamps) return fail(ctx, ENTWINE_EUNSUPPORTED, "the call has no workgroup timestamps");
  if (nwgs) *nwgs = s.grid;
  if (nproducers) *nproducers = s.G;
  if (ticks_per_us) *ticks_per_us = double(ctx->ticks_per_us);
  if (!stamps) return ENTWINE_OK;
  if (capacity < s.grid * 4) return fail(ctx, ENTWINE_EINVAL, "capacity below %d", s.grid * 4);
  std::vector<unsigned long long> h;
  CHECK(read_stamps(ctx, s, h));
  for (int b = 0; b < s.grid; ++b)
    for (int i = 0; i < 4; ++i) stamps[4 * b + i] = h[size_t(kStampsPerWg) * b + i];
  return ENTWINE_OK;
}

entwine_status entwine_last_clock(entwine_ctx* ctx, int32_t back, double* ghz) {
  if (!ctx) return fail(nullptr, ENTWINE_EINVAL, "ctx is NULL");
  if (!ghz) return fail(ctx, ENTWINE_EINVAL, "ghz is NULL");
  if (back < 0 || back >= kRing || back >= ctx->ncalls) return fail(ctx, ENTWINE_EINVAL, "no such timed call");
  const TimingSlot& s = ctx->ring[(ctx->ncalls - 1 - back) % kRing];
  if (!s.has_stamps) return fail(ctx, ENTWINE_EUNSUPPORTED, "the call has no workgroup timestamps");
  std::vector<unsigned long long> h;
  CHECK(read_stamps(ctx, s, h));
  // Cycles over wall-clock time, summed over the producer workgroups.
  double cycles = 0.0, ticks = 0.0;
  for (int b = 0; b < s.G; ++b) {
    const unsigned long long* t = h.data() + size_t(kStampsPerWg) * b;
    if (t[1] <= t[0] || t[5] <= t[4]) continue;
    cycles += double(t[5] - t[4]);
    ticks += double(t[1] - t[0]);
  }
  *ghz = ticks > 0.0 ? cycles / (ticks / double(ctx->ticks_per_us)) / 1e3 : 0.0;
  return ENTWINE_OK;
}

entwine_status entwine_tile_schedule(int32_t order, int64_t M, int64_t N, int32_t P, int32_t BM, int32_t BN,
                                     int32_t group_m, int32_t* blocks, int32_t* tiles) {
  CHECK(validate_shape(nullptr, M, N, 8, P));
  if (order < 0 || order > 2) return fail(nullptr, ENTWINE_EINVAL, "unknown order");
  if (BM <= 0 || BN <= 0 || BM % ENTWINE_TILE || BN % ENTWINE_TILE || (M / P) % BM || N % BN)
    return fail(nullptr, ENTWINE_EUNSUPPORTED, "block shape does not tile the chunk");
  if (group_m < 0 || group_m > 64) return fail(nullptr, ENTWINE_EINVAL, "group_m outside [0, 64]");
  const BlockGrid g = make_grid(int(M), int(N), P, BM, BN, group_m);
  const int nb = g.MB * g.NB;
  const int tiles_n = int(N / ENTWINE_TILE);
  for (int p = 0; p < nb; ++p) {
    const BlockPos b = block_of_position(order, p, g);
    if (blocks) {
      blocks[4 * p + 0] = b.d;
      blocks[4 * p + 1] = b.l;
      blocks[4 * p + 2] = b.mb;
      blocks[4 * p + 3] = b.nb;
    }
  }
  if (tiles) {
    const int Q = tiles_per_partition(int(M), int(N), P);
    for (int d = 0; d < P; ++d)
      for (int t = 0; t < Q; ++t) {
        int tr, tc;
        tile_of_number(d, t, g, &tr, &tc);
        tiles[2 * (tr * tiles_n + tc) + 0] = d;
        tiles[2 * (tr * tiles_n + tc) + 1] = t;
      }
  }
  return ENTWINE_OK;
}

entwine_status entwine_consumer_tasks(int32_t dest, int32_t P, int32_t Q, int32_t x, int32_t j, int32_t* part,
                                      int32_t* tasks, int32_t cap, int32_t* count) {
  if (P < 1 || Q < 0 || x < 1 || j < 0 || j >= x) return fail(nullptr, ENTWINE_EINVAL, "bad consumer arguments");
  if (dest == ENTWINE_DEST_ALL && x % P) return fail(nullptr, ENTWINE_EINVAL, "x must be a multiple of P");
  const ConsumerSeq s = consumer_seq(dest, P, x, j);
  int n = 0;
  for (int t = s.first; t < Q; t += s.stride) {
    if (tasks && n < cap) tasks[n] = t;
    ++n;
  }
  if (part) *part = s.part;
  if (count) *count = n;
  return ENTWINE_OK;
}

}  // extern "C"
