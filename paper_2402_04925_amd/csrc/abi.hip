// extern "C" entry points of libtpdq: argument validation, workspace layout
// and dispatch to the gfx950 kernels. Nothing here touches tensor data on the
// host; every step of the computation runs in the kernels.
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "tpdq_internal.h"

using namespace tpdq;

// Scratch of tpdq_mlp_shard_noalloc: a workspace owned by the library for
// callers that cannot allocate device memory. Every GPU the library runs on
// holds its own copy from the time the code object is loaded until the
// process ends. In host code `scratch` is only a stand-in for the symbol:
// the device address of a GPU's copy comes from hipGetSymbolAddress, taken
// once per device with that device current (scratch_ptr), and only that
// address is ever handed to a kernel or a copy.
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

thread_local std::string g_last_error;

tpdq_status fail(tpdq_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

tpdq_status hip_fail(hipError_t e, const char* what) {
  return fail(TPDQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Shape and pointer checks of one layer. `need_gidx`: the act-order path
// reads g_idx; `sorted`: the rows are sorted by group, so with G > 0 the group
// of row k is k / G (the last group may be partial) and num_groups must cover
// ceil(K / G); with G == 0 (groups of unequal sizes) the sorted g_idx gives
// each row's group and is required.
tpdq_status check_layer(const tpdq_w4* w, const char* name, bool need_gidx, bool sorted) {
  if (!w) return fail(TPDQ_ERR_NULL, "%s is NULL", name);
  if (!w->qweight || !w->scales || !w->qzeros)
    return fail(TPDQ_ERR_NULL, "%s: qweight, scales and qzeros are required", name);
  if (need_gidx && !w->g_idx) return fail(TPDQ_ERR_NULL, "%s: g_idx is required", name);
  if (w->K <= 0 || w->N <= 0 || w->group_size < 0 || w->num_groups <= 0)
    return fail(TPDQ_ERR_SHAPE, "%s: K=%d N=%d num_groups=%d must be positive, G=%d not negative",
                name, w->K, w->N, w->num_groups, w->group_size);
  if (w->K % 8 || w->N % 8 || w->group_size % 8)
    return fail(TPDQ_ERR_SHAPE, "%s: K=%d, N=%d and G=%d must be multiples of 8", name, w->K, w->N,
                w->group_size);
  if (w->zero_offset != 0 && w->zero_offset != 1)
    return fail(TPDQ_ERR_SHAPE, "%s: zero_offset=%d must be 0 or 1", name, w->zero_offset);
  if (sorted) {
    if (w->group_size == 0 && !w->g_idx)
      return fail(TPDQ_ERR_NULL, "%s: sorted rows in groups of unequal sizes (G = 0) need their g_idx",
                  name);
    const int ngk = w->group_size ? (w->K + w->group_size - 1) / w->group_size : 1;
    if (w->num_groups < ngk)
      return fail(TPDQ_ERR_SHAPE, "%s: num_groups=%d < ceil(K/G)=%d", name, w->num_groups, ngk);
  }
  if (w->layout != TPDQ_LAYOUT_GPTQ && w->layout != TPDQ_LAYOUT_TILED)
    return fail(TPDQ_ERR_SHAPE, "%s: unknown layout %d", name, w->layout);
  const int64_t ldq_min = w->layout == TPDQ_LAYOUT_TILED ? tiled_ld(w->K) : (int64_t)w->N;
  if (w->ld_q < ldq_min || w->ld_s < w->N || w->ld_z < w->N / 8)
    return fail(TPDQ_ERR_SHAPE, "%s: leading dimensions too small (ld_q=%lld ld_s=%lld ld_z=%lld)",
                name, (long long)w->ld_q, (long long)w->ld_s, (long long)w->ld_z);
  // the kernels address each tensor through a buffer resource with 32-bit
  // byte offsets
  const int64_t lim = (int64_t)1 << 31;
  const int64_t qrows = w->layout == TPDQ_LAYOUT_TILED ? (int64_t)(w->N + 15) / 16 : w->K / 8;
  if (qrows * w->ld_q * 4 >= lim || (int64_t)w->num_groups * w->ld_s * 2 >= lim ||
      (int64_t)w->num_groups * w->ld_z * 4 >= lim)
    return fail(TPDQ_ERR_UNSUPPORTED, "%s: qweight, scales or qzeros spans 2 GiB or more", name);
  if (!aligned(w->qweight, 16) || w->ld_q % 4)
    return fail(TPDQ_ERR_ALIGN, "%s: qweight needs 16-byte alignment and ld_q %% 4 == 0", name);
  if (!aligned(w->scales, 8) || w->ld_s % 4)
    return fail(TPDQ_ERR_ALIGN, "%s: scales need 8-byte alignment and ld_s %% 4 == 0", name);
  if (!aligned(w->qzeros, 4)) return fail(TPDQ_ERR_ALIGN, "%s: qzeros need 4-byte alignment", name);
  if (need_gidx && !aligned(w->g_idx, 16))
    return fail(TPDQ_ERR_ALIGN, "%s: g_idx needs 16-byte alignment", name);
  return TPDQ_OK;
}

// Workspace of one GEMM call. The decode kernels use it only for the
// gathered activations when the gather X[:, perm] cannot be done inside the
// GEMM's LDS: the prepared operand (k_gather_prep: 16 rows x 128 columns x
// 2 bytes per row tile and 128-row block, chunks of 64 rows). The M-tiled
// kernel uses [X[:, perm] row-major, M x K x 2 bytes, when perm is given]
// [fp32 split-K partials].
size_t decode_gather_bytes(int M, int K) {
  const int mc = std::min(M, kDecodeMaxM);
  return align_up((size_t)((mc + kTileM - 1) / kTileM) * ((K + 127) / 128) * 4096);
}

size_t mtile_gather_bytes(int M, int K, bool perm) { return perm ? align_up((size_t)M * K * 2) : 0; }

// The M-tiled kernel's plan when it covers the call. With a perm its row
// gather (k_gather_rows) stages one row of X, K halves, in LDS: past that the
// call runs through the decode kernels, whose gathers have no such limit.
bool mtile_for(int M, int64_t ldx, bool perm, const tpdq_w4* w, int meta, MtilePlan* p) {
  if (perm && (size_t)w->K * 2 > kLdsMax) return false;
  return plan_mtile(M, perm ? (int64_t)w->K : ldx, w, meta, p);
}

// The decode plan of one launch of mc <= 64 rows, as run_gemm makes it: with
// a perm, the gather inside the kernel's LDS if it is planned; else, up to 4
// rows, X' gathered once row-major when the tile kernel then takes it like
// any X (*plain); else the prepared operand (*prepared). The workspace of the
// prepared operand is at least that of the row-major X', so sizes computed
// without `plain` cover both.
bool decode_plan_for(int mc, bool perm, const tpdq_w4* w, int meta, int dt, DecodePlan* plan,
                     bool* prepared, bool gated = false, bool* plain = nullptr) {
  *prepared = false;
  if (plain) *plain = false;
  if (perm) {
    if (plan_decode(mc, w->K, w->N, w->group_size, w->num_groups, w->layout, meta, kOperandGather,
                    dt, plan, gated))
      return true;
    if (plain && mc <= 4 &&
        plan_decode(mc, w->K, w->N, w->group_size, w->num_groups, w->layout, meta, kOperandPlain, dt,
                    plan, gated) &&
        !plan->wide) {
      *plain = true;
      return true;
    }
    *prepared = true;
    return plan_decode(mc, w->K, w->N, w->group_size, w->num_groups, w->layout, meta,
                       kOperandPrepared, dt, plan, gated);
  }
  return plan_decode(mc, w->K, w->N, w->group_size, w->num_groups, w->layout, meta, kOperandPlain,
                     dt, plan, gated);
}

// split-K partials of the wide decode kernel (0 when K is not split)
size_t decode_part_bytes(const DecodePlan& p, int mc, int N) {
  return p.wide && p.ks > 1 ? align_up((size_t)p.ks * mc * N * 4) : 0;
}

// Bytes the call (X with leading dimension ldx, optional perm) uses. Decode:
// [prepared operand][wide kernel's partials], the partials after the
// prepared-operand region whenever either is used. The plans, and so the
// bytes, are the same for both element types.
// The gated GEMM (gated = true) runs the decode kernels only.
size_t gemm_ws_need(int M, int64_t ldx, bool perm, const tpdq_w4* w, int meta, int dt = TPDQ_FP16,
                    bool gated = false) {
  MtilePlan p;
  if (!gated && mtile_for(M, ldx, perm, w, meta, &p))
    return mtile_gather_bytes(M, w->K, perm) + mtile_part_bytes(p, M, w->N);
  DecodePlan dp;
  bool prepared = false;
  const int mc = std::min(M, kDecodeMaxM);  // the largest launch
  if (!decode_plan_for(mc, perm, w, meta, dt, &dp, &prepared, gated))
    return perm ? decode_gather_bytes(M, w->K) : 0;
  const size_t part = decode_part_bytes(dp, mc, w->N);
  return (prepared || part ? decode_gather_bytes(M, w->K) : 0) + part;
}

int meta_mode(tpdq_path path) {
  if (path == TPDQ_PATH_ORDERED) return kMetaGroup;
  if (path == TPDQ_PATH_ACTORDER_GLOBAL) return kMetaRowGlobal;
  return kMetaRowLds;
}

// Extra inputs and outputs of one GEMM inside the MLP (decode kernels, one
// launch of M <= 64 rows): yp receives a second copy of Y in the prepared
// operand layout of the next GEMM; x_prepared says X already is one.
struct GemmIO {
  uint16_t* yp = nullptr;
  int yp_natural = 0;
  bool x_prepared = false;
  const tpdq_w4* up = nullptr;  // gated GEMM: Y = silu(X' W) * (X' W_up), decode kernels only
};

// One GEMM through the decode kernels, M cut into launches of <= 64 rows.
// perm != NULL: the operand is X[:, perm]; it is gathered inside the kernel
// when it fits in LDS, else into the workspace first (already in operand
// order).
tpdq_status run_gemm(const uint16_t* X, int64_t ldx, int M, const int32_t* perm, const tpdq_w4* w,
                     tpdq_path path, int dt, uint16_t* Y, int64_t ldy, char* ws, hipStream_t st,
                     const GemmIO& io = GemmIO()) {
  const int meta = meta_mode(path);
  // sorted rows in groups of G read no g_idx; in groups of unequal sizes their
  // sorted g_idx gives each row's group (the per-row kernel, on sorted rows)
  const int32_t* gidx = path == TPDQ_PATH_ORDERED && w->group_size > 0 ? nullptr : w->g_idx;
  MtilePlan mp;
  const bool gated = io.up != nullptr;
  if (!gated && mtile_for(M, ldx, perm != nullptr, w, meta, &mp)) {
    // M-tiled MFMA GEMM over all rows, the activations gathered first
    const uint16_t* Xa = X;
    int64_t lda = ldx;
    if (perm) {
      uint16_t* Xp = (uint16_t*)ws;
      hipError_t e = launch_gather_rows(X, ldx, M, w->K, perm, Xp, st);
      if (e != hipSuccess) return hip_fail(e, "activation gather launch");
      Xa = Xp;
      lda = w->K;
    }
    GemmArgs a{};
    a.X = Xa;
    a.ldx = lda;
    a.M = M;
    a.qw = (const uint32_t*)w->qweight;
    a.ldq = w->ld_q;
    a.sc = (const uint16_t*)w->scales;
    a.lds = w->ld_s;
    a.qz = (const uint32_t*)w->qzeros;
    a.ldz = w->ld_z;
    a.K = w->K;
    a.N = w->N;
    a.G = w->group_size;
    a.num_groups = w->num_groups;
    a.zoff = w->zero_offset;
    a.dt = dt;
    a.Y = Y;
    a.ldy = ldy;
    float* part = (float*)(ws + mtile_gather_bytes(M, w->K, perm != nullptr));
    hipError_t e = launch_mtile(a, mp, part, st);
    if (e != hipSuccess) return hip_fail(e, "M-tiled GEMM launch");
    return TPDQ_OK;
  }
  for (int m0 = 0; m0 < M; m0 += kDecodeMaxM) {
    const int mc = std::min(kDecodeMaxM, M - m0);
    const uint16_t* Xc = X + (int64_t)m0 * ldx;
    int64_t ldc = ldx;
    DecodePlan plan;
    bool prepared = false, plain = false;
    const bool ok = io.x_prepared
                        ? plan_decode(mc, w->K, w->N, w->group_size, w->num_groups, w->layout, meta,
                                      kOperandPrepared, dt, &plan, gated)
                        : decode_plan_for(mc, perm != nullptr, w, meta, dt, &plan, &prepared, gated,
                                          &plain);
    const int operand =
        perm ? (prepared ? kOperandPrepared : (plain ? kOperandPlain : kOperandGather)) : kOperandPlain;
    if (ok && plain) {
      uint16_t* Xp = (uint16_t*)ws;
      hipError_t e = launch_gather_plain(Xc, ldx, mc, w->K, perm, Xp, st);
      if (e != hipSuccess) return hip_fail(e, "activation gather launch");
      Xc = Xp;
      ldc = w->K;
    }
    if (ok && prepared) {
      uint16_t* Xp = (uint16_t*)ws;
      hipError_t e = launch_gather_prep(Xc, ldx, mc, w->K, perm, w->layout, Xp, st);
      if (e != hipSuccess) return hip_fail(e, "activation gather launch");
      Xc = Xp;
      ldc = w->K;
    }
    if (!ok)
      return fail(TPDQ_ERR_UNSUPPORTED, "no decode kernel for M=%d K=%d N=%d G=%d", mc, w->K, w->N,
                  w->group_size);
    GemmArgs a{};
    a.X = Xc;
    a.ldx = ldc;
    a.M = mc;
    a.perm = operand == kOperandGather ? perm : nullptr;
    a.qw = (const uint32_t*)w->qweight;
    a.ldq = w->ld_q;
    a.sc = (const uint16_t*)w->scales;
    a.lds = w->ld_s;
    a.qz = (const uint32_t*)w->qzeros;
    a.ldz = w->ld_z;
    a.g_idx = gidx;
    a.K = w->K;
    a.N = w->N;
    a.G = w->group_size;
    a.num_groups = w->num_groups;
    a.zoff = w->zero_offset;
    a.dt = dt;
    a.Y = Y + (int64_t)m0 * ldy;
    a.ldy = ldy;
    a.Yp = io.yp;
    a.yp_natural = io.yp_natural;
    if (gated) {
      a.qw_up = (const uint32_t*)io.up->qweight;
      a.sc_up = (const uint16_t*)io.up->scales;
      a.qz_up = (const uint32_t*)io.up->qzeros;
    }
    float* part = (float*)(ws + decode_gather_bytes(M, w->K));
    hipError_t e = launch_decode(a, plan, part, st);
    if (e != hipSuccess) return hip_fail(e, "decode GEMM launch");
  }
  return TPDQ_OK;
}

bool is_actorder(tpdq_path p) { return p == TPDQ_PATH_ACTORDER || p == TPDQ_PATH_ACTORDER_GLOBAL; }

// The MLP's GEMM2 reads Y1 from global memory when Y1 does not fit in LDS;
// row-major, every load of 16 rows touches 16 rows a row apart (address
// translation and L1 tag stalls), so GEMM1 then also writes Y1 in GEMM2's
// operand order (one contiguous KiB per load) into the workspace. Both
// GEMMs must be single decode launches of the tile kernels (not k_wide, not
// the M-tiled kernel), and N1 a multiple of 128 (no padding to fill).
bool mlp_prepared_y1(int M, int64_t ldx, bool perm, const tpdq_w4* w1, const tpdq_w4* w2, int meta,
                     int dt, bool gated = false) {
  if (M > kDecodeMaxM || w1->N % 128 != 0) return false;
  MtilePlan mp;
  if ((!gated && mtile_for(M, ldx, perm, w1, meta, &mp)) ||
      plan_mtile(M, w1->N, w2, meta, &mp))
    return false;
  DecodePlan p1, p2;
  bool prepared = false;
  if (!decode_plan_for(M, perm, w1, meta, dt, &p1, &prepared, gated) || p1.wide) return false;
  // GEMM2 would read row-major Y1 from global memory: through the tile
  // kernel, or through k_wide only because of the row-major rule (on
  // weights of kWideMinWeights or more GEMM2 stays on k_wide instead)
  const bool big2 = (int64_t)w2->K * w2->N >= kWideMinWeights;
  if (!decode_plan_for(M, false, w2, meta, dt, &p2, &prepared) || (p2.wide && big2) ||
      p2.amode != kAGlobal)
    return false;
  DecodePlan p3;
  return plan_decode(M, w2->K, w2->N, w2->group_size, w2->num_groups, w2->layout, meta,
                     kOperandPrepared, dt, &p3) && !p3.wide;
}

// The device address of each GPU's copy of `scratch`, taken once per device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// The device address of the scratch copy of the stream's GPU.
tpdq_status scratch_ptr(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "device of the stream");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(TPDQ_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return hip_fail(e, "hipSetDevice");
    void* p = nullptr;
    const hipError_t es = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev && (e = hipSetDevice(cur)) != hipSuccess) return hip_fail(e, "hipSetDevice");
    if (es != hipSuccess) return hip_fail(es, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(TPDQ_ERR_HIP, "hipGetSymbolAddress(scratch) gave NULL");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return TPDQ_OK;
}

tpdq_status check_common(int32_t M, tpdq_path path, tpdq_dtype dtype) {
  if (M < 1) return fail(TPDQ_ERR_SHAPE, "M=%d must be >= 1", M);
  if (path != TPDQ_PATH_ACTORDER && path != TPDQ_PATH_ORDERED && path != TPDQ_PATH_ACTORDER_GLOBAL)
    return fail(TPDQ_ERR_SHAPE, "unknown path %d", (int)path);
  if (dtype != TPDQ_FP16 && dtype != TPDQ_BF16) return fail(TPDQ_ERR_SHAPE, "unknown dtype %d", (int)dtype);
  return TPDQ_OK;
}

}  // namespace

extern "C" {

const char* tpdq_version(void) { return "0.1.0"; }

const char* tpdq_status_string(tpdq_status s) {
  switch (s) {
    case TPDQ_OK: return "ok";
    case TPDQ_ERR_NULL: return "null pointer";
    case TPDQ_ERR_SHAPE: return "invalid shape";
    case TPDQ_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case TPDQ_ERR_GIDX: return "invalid g_idx";
    case TPDQ_ERR_WORKSPACE: return "workspace too small";
    case TPDQ_ERR_UNSUPPORTED: return "unsupported";
    case TPDQ_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* tpdq_last_error(void) { return g_last_error.c_str(); }

size_t tpdq_workspace_bytes(int op, int32_t M, const tpdq_w4* a, const tpdq_w4* b) {
  if (!a || a->K <= 0 || a->N <= 0 || a->group_size < 0 || a->num_groups <= 0) return 0;
  if (op == 0) {
    size_t n = 256 + align_up((size_t)a->num_groups * 4);
    if (b) n += align_up((size_t)b->num_groups * 4);
    return n;
  }
  if (M < 1) return 0;
  // the most any call of this shape can use (the leading dimension of X is
  // not known here; ldx = K is the case that can take the M-tiled kernel)
  auto gemm_max = [&](const tpdq_w4* w, bool perm_possible) {
    size_t n = perm_possible ? decode_gather_bytes(M, w->K) : 0;
    for (int pm = 0; pm <= (perm_possible ? 1 : 0); ++pm)
      for (int meta : {kMetaGroup, kMetaRowLds, kMetaRowGlobal})
        n = std::max(n, gemm_ws_need(M, w->K, pm == 1, w, meta));
    return n;
  };
  if (op == 1) return gemm_max(a, true);
  if (op == 2 || op == 3) {
    if (!b) return 0;
    // GEMM1's region, then Y1 in GEMM2's operand order (mlp_prepared_y1);
    // op 3: GEMM1 is the gated GEMM (a = w_gate)
    const size_t y1p = M <= kDecodeMaxM ? decode_gather_bytes(M, a->N) : 0;
    size_t g1 = gemm_max(a, true);
    if (op == 3) {
      g1 = decode_gather_bytes(M, a->K);
      for (int pm = 0; pm <= 1; ++pm)
        for (int meta : {kMetaGroup, kMetaRowLds, kMetaRowGlobal})
          g1 = std::max(g1, gemm_ws_need(M, a->K, pm == 1, a, meta, TPDQ_FP16, true));
    }
    return std::max(g1 + y1p, gemm_max(b, false));
  }
  return 0;
}

tpdq_status tpdq_reorder(const tpdq_w4* w1, const tpdq_w4* w2, int32_t* P1, int32_t* g1_sorted,
                         int32_t* P2, int32_t* g2_sorted, int32_t* qweight1_out,
                         void* scales1_out, int32_t* qzeros1_out, int32_t* qweight2_out,
                         tpdq_dtype dtype, tpdq_layout out_layout, void* workspace,
                         size_t ws_bytes, void* stream) {
  tpdq_status st = check_layer(w1, "w1", true, false);
  if (st != TPDQ_OK) return st;
  if (w1->layout != TPDQ_LAYOUT_GPTQ || (w2 && w2->layout != TPDQ_LAYOUT_GPTQ))
    return fail(TPDQ_ERR_SHAPE, "reorder takes GPTQ-layout inputs");
  if (out_layout != TPDQ_LAYOUT_GPTQ && out_layout != TPDQ_LAYOUT_TILED)
    return fail(TPDQ_ERR_SHAPE, "unknown output layout %d", (int)out_layout);
  if (dtype != TPDQ_FP16 && dtype != TPDQ_BF16) return fail(TPDQ_ERR_SHAPE, "unknown dtype");
  // Eq. 3 over a whole layer: ceil(K/G) groups; groups of unequal sizes (G == 0)
  // come with their own count
  auto global_groups_ok = [](const tpdq_w4* w) {
    return w->group_size == 0 || w->num_groups == (w->K + w->group_size - 1) / w->group_size;
  };
  if (!global_groups_ok(w1))
    return fail(TPDQ_ERR_SHAPE, "w1: a global act-order layer has num_groups == ceil(K/G)");
  if (!P1 || !g1_sorted || !qweight1_out || !scales1_out || !qzeros1_out)
    return fail(TPDQ_ERR_NULL, "P1, g1_sorted, qweight1_out, scales1_out, qzeros1_out are required");
  if (w2) {
    st = check_layer(w2, "w2", true, false);
    if (st != TPDQ_OK) return st;
    if (w2->K != w1->N) return fail(TPDQ_ERR_SHAPE, "w2->K=%d != w1->N=%d", w2->K, w1->N);
    if (!global_groups_ok(w2))
      return fail(TPDQ_ERR_SHAPE, "w2: a global act-order layer has num_groups == ceil(K/G)");
    if (!P2 || !g2_sorted || !qweight2_out)
      return fail(TPDQ_ERR_NULL, "P2, g2_sorted and qweight2_out are required with w2");
  } else if (P2 || g2_sorted || qweight2_out) {
    return fail(TPDQ_ERR_SHAPE, "P2, g2_sorted and qweight2_out must be NULL without w2");
  }
  const size_t need = tpdq_workspace_bytes(0, 0, w1, w2);
  if (!workspace || ws_bytes < need)
    return fail(TPDQ_ERR_WORKSPACE, "reorder needs %zu workspace bytes, got %zu", need, ws_bytes);
  if (!aligned(workspace, 16)) return fail(TPDQ_ERR_ALIGN, "workspace needs 16-byte alignment");

  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  uint32_t* flags = (uint32_t*)ws;  // [0] w1, [1] w2
  uint32_t* counts1 = (uint32_t*)(ws + 256);
  uint32_t* counts2 = (uint32_t*)(ws + 256 + align_up((size_t)w1->num_groups * 4));
  const size_t nwords = need / 4;
  hipError_t e = launch_fill_u32((uint32_t*)ws, nwords, 0u, s);
  if (e != hipSuccess) return hip_fail(e, "workspace clear");

  ReorderLayer L1{w1->g_idx, w1->K, w1->group_size, w1->num_groups, P1, g1_sorted};
  ReorderLayer L2{};
  e = launch_gidx_validate(L1, counts1, flags + 0, s);
  if (e != hipSuccess) return hip_fail(e, "g_idx validation launch");
  if (w2) {
    L2 = ReorderLayer{w2->g_idx, w2->K, w2->group_size, w2->num_groups, P2, g2_sorted};
    e = launch_gidx_validate(L2, counts2, flags + 1, s);
    if (e != hipSuccess) return hip_fail(e, "g_idx validation launch");
  }
  uint32_t hflags[2] = {0, 0};
  e = hipMemcpyAsync(hflags, flags, sizeof(hflags), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "g_idx validation readback");
  for (int l = 0; l < 2; ++l) {
    if (hflags[l] & 1u)
      return fail(TPDQ_ERR_GIDX, "w%d: a g_idx value is outside [0, num_groups)", l + 1);
    if (hflags[l] & 2u)
      return fail(TPDQ_ERR_GIDX, "w%d: the groups do not hold the rows Eq. 3 gives (G each, the last "
                  "K - (num_groups - 1) G)", l + 1);
  }

  e = launch_gidx_rank(L1, counts1, s);
  if (e == hipSuccess && w2) e = launch_gidx_rank(L2, counts2, s);
  if (e != hipSuccess) return hip_fail(e, "argsort launch");

  const int32_t* pcol = w2 ? P2 : nullptr;
  const int ng1 = w1->num_groups;
  e = launch_permute_qweight((const uint32_t*)w1->qweight, w1->ld_q, w1->K, w1->N, P1, pcol,
                             (uint32_t*)qweight1_out, out_layout, s);
  if (e == hipSuccess)
    e = launch_permute_scales((const uint16_t*)w1->scales, w1->ld_s, ng1, w1->N, pcol,
                              (uint16_t*)scales1_out, s);
  if (e == hipSuccess)
    e = launch_permute_qzeros((const uint32_t*)w1->qzeros, w1->ld_z, ng1, w1->N, pcol,
                              (uint32_t*)qzeros1_out, s);
  if (e == hipSuccess && w2)
    e = launch_permute_qweight((const uint32_t*)w2->qweight, w2->ld_q, w2->K, w2->N, P2, nullptr,
                               (uint32_t*)qweight2_out, out_layout, s);
  if (e != hipSuccess) return hip_fail(e, "permute launch");
  return TPDQ_OK;
}

tpdq_status tpdq_pack_tiled(const tpdq_w4* w, int32_t* qweight_out, void* stream) {
  if (!w) return fail(TPDQ_ERR_NULL, "w is NULL");
  if (!w->qweight || !qweight_out) return fail(TPDQ_ERR_NULL, "qweight and qweight_out are required");
  if (w->layout != TPDQ_LAYOUT_GPTQ) return fail(TPDQ_ERR_SHAPE, "input must be GPTQ layout");
  if (w->K <= 0 || w->N <= 0 || w->K % 8 || w->N % 8)
    return fail(TPDQ_ERR_SHAPE, "K=%d and N=%d must be positive multiples of 8", w->K, w->N);
  if (w->ld_q < w->N) return fail(TPDQ_ERR_SHAPE, "ld_q=%lld < N=%d", (long long)w->ld_q, w->N);
  if (!aligned(qweight_out, 16)) return fail(TPDQ_ERR_ALIGN, "qweight_out needs 16-byte alignment");
  hipError_t e = launch_permute_qweight((const uint32_t*)w->qweight, w->ld_q, w->K, w->N, nullptr,
                                        nullptr, (uint32_t*)qweight_out, TPDQ_LAYOUT_TILED,
                                        (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "pack launch");
  return TPDQ_OK;
}

tpdq_status tpdq_w4a16_gemm(const void* X, int64_t ldx, int32_t M, const int32_t* x_perm,
                            const tpdq_w4* w, tpdq_path path, tpdq_dtype dtype, void* Y,
                            int64_t ldy, void* workspace, size_t ws_bytes, void* stream) {
  tpdq_status st = check_common(M, path, dtype);
  if (st != TPDQ_OK) return st;
  st = check_layer(w, "w", is_actorder(path), path == TPDQ_PATH_ORDERED);
  if (st != TPDQ_OK) return st;
  if (!X || !Y) return fail(TPDQ_ERR_NULL, "X and Y are required");
  if (ldx < w->K || ldy < w->N)
    return fail(TPDQ_ERR_SHAPE, "ldx=%lld < K=%d or ldy=%lld < N=%d", (long long)ldx, w->K,
                (long long)ldy, w->N);
  // every path reads X (gathered or not) with 16-byte vector loads of row m at
  // column 8r
  if (!aligned(X, 16) || ldx % 8)
    return fail(TPDQ_ERR_ALIGN, "X needs 16-byte alignment and ldx %% 8 == 0");
  if (!aligned(Y, 8) || ldy % 4) return fail(TPDQ_ERR_ALIGN, "Y needs 8-byte alignment, ldy %% 4 == 0");
  // a call that uses a workspace (a gather always does) takes the documented
  // tpdq_workspace_bytes(1, ...), an upper bound of what it uses
  const size_t bound = tpdq_workspace_bytes(1, M, w, nullptr);
  const size_t need = gemm_ws_need(M, ldx, x_perm != nullptr, w, meta_mode(path), dtype);
  if ((x_perm || need) && (!workspace || ws_bytes < bound))
    return fail(TPDQ_ERR_WORKSPACE, "GEMM needs %zu workspace bytes, got %zu", bound, ws_bytes);
  if (workspace && !aligned(workspace, 16))
    return fail(TPDQ_ERR_ALIGN, "workspace needs 16-byte alignment");
  return run_gemm((const uint16_t*)X, ldx, M, x_perm, w, path, dtype, (uint16_t*)Y, ldy,
                  (char*)workspace, (hipStream_t)stream);
}

}  // extern "C"

namespace {

// tpdq_mlp_shard, with the caller's workspace or (noalloc) the library's
// scratch: every argument is validated first; the scratch address is taken
// only after that.
tpdq_status mlp_shard(const void* X, int64_t ldx, int32_t M, const int32_t* P1, const tpdq_w4* w1,
                      const tpdq_w4* w2, tpdq_path path, tpdq_dtype dtype, void* Y1,
                      void* Y2_partial, void* workspace, size_t ws_bytes, void* stream,
                      bool noalloc) {
  tpdq_status st = check_common(M, path, dtype);
  if (st != TPDQ_OK) return st;
  const bool act = is_actorder(path);
  st = check_layer(w1, "w1", act, !act);
  if (st != TPDQ_OK) return st;
  st = check_layer(w2, "w2", act, !act);
  if (st != TPDQ_OK) return st;
  if (w2->K != w1->N) return fail(TPDQ_ERR_SHAPE, "w2->K=%d != w1->N=%d", w2->K, w1->N);
  if (!X || !Y1 || !Y2_partial) return fail(TPDQ_ERR_NULL, "X, Y1 and Y2_partial are required");
  if (act && P1) return fail(TPDQ_ERR_SHAPE, "the act-order paths take no P1");
  if (!act && !P1) return fail(TPDQ_ERR_NULL, "the ordered path needs P1");
  if (ldx < w1->K) return fail(TPDQ_ERR_SHAPE, "ldx=%lld < K1=%d", (long long)ldx, w1->K);
  if (!aligned(X, 16) || ldx % 8)
    return fail(TPDQ_ERR_ALIGN, "X needs 16-byte alignment and ldx %% 8 == 0");
  if (!aligned(Y1, 16) || !aligned(Y2_partial, 8))
    return fail(TPDQ_ERR_ALIGN, "Y1 needs 16-byte and Y2_partial 8-byte alignment");
  const int meta = meta_mode(path);
  const size_t bound = tpdq_workspace_bytes(2, M, w1, w2);
  const size_t need = std::max(gemm_ws_need(M, ldx, !act, w1, meta, dtype),
                               gemm_ws_need(M, w1->N, false, w2, meta, dtype));
  if (noalloc) {
    if (bound > kScratchBytes)
      return fail(TPDQ_ERR_WORKSPACE,
                  "MLP needs %zu bytes of scratch; the library's static scratch holds %zu "
                  "(use tpdq_mlp_shard with a workspace)", bound, kScratchBytes);
    st = scratch_ptr((hipStream_t)stream, &workspace);
    if (st != TPDQ_OK) return st;
    ws_bytes = kScratchBytes;
  }
  if ((!act || need) && (!workspace || ws_bytes < bound))
    return fail(TPDQ_ERR_WORKSPACE, "MLP needs %zu workspace bytes, got %zu", bound, ws_bytes);
  if (workspace && !aligned(workspace, 16))
    return fail(TPDQ_ERR_ALIGN, "workspace needs 16-byte alignment");

  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  GemmIO io1, io2;
  if (workspace && ws_bytes >= bound && mlp_prepared_y1(M, ldx, !act, w1, w2, meta, dtype)) {
    const size_t off = gemm_ws_need(M, ldx, !act, w1, meta, dtype);
    io1.yp = (uint16_t*)(ws + off);
    io1.yp_natural = w2->layout == TPDQ_LAYOUT_TILED ? 1 : 0;
    io2.x_prepared = true;
  }
  st = run_gemm((const uint16_t*)X, ldx, M, act ? nullptr : P1, w1, path, dtype, (uint16_t*)Y1, w1->N,
                ws, s, io1);
  if (st != TPDQ_OK) return st;
  if (io2.x_prepared)
    return run_gemm(io1.yp, w1->N, M, nullptr, w2, path, dtype, (uint16_t*)Y2_partial, w2->N, ws, s,
                    io2);
  return run_gemm((const uint16_t*)Y1, w1->N, M, nullptr, w2, path, dtype, (uint16_t*)Y2_partial,
                  w2->N, ws, s);
}

}  // namespace

extern "C" {

tpdq_status tpdq_mlp_shard(const void* X, int64_t ldx, int32_t M, const int32_t* P1,
                           const tpdq_w4* w1, const tpdq_w4* w2, tpdq_path path, tpdq_dtype dtype,
                           void* Y1, void* Y2_partial, void* workspace, size_t ws_bytes,
                           void* stream) {
  return mlp_shard(X, ldx, M, P1, w1, w2, path, dtype, Y1, Y2_partial, workspace, ws_bytes, stream,
                   false);
}

tpdq_status tpdq_mlp_shard_noalloc(const void* X, int64_t ldx, int32_t M, const int32_t* P1,
                                   const tpdq_w4* w1, const tpdq_w4* w2, tpdq_path path,
                                   tpdq_dtype dtype, void* Y1, void* Y2_partial, void* stream) {
  return mlp_shard(X, ldx, M, P1, w1, w2, path, dtype, Y1, Y2_partial, nullptr, 0, stream, true);
}

tpdq_status tpdq_gated_mlp_shard(const void* X, int64_t ldx, int32_t M, const int32_t* P1,
                                 const tpdq_w4* w_gate, const tpdq_w4* w_up, const tpdq_w4* w_down,
                                 tpdq_path path, tpdq_dtype dtype, void* Y1, void* Y2_partial,
                                 void* workspace, size_t ws_bytes, void* stream) {
  tpdq_status st = check_common(M, path, dtype);
  if (st != TPDQ_OK) return st;
  const bool act = is_actorder(path);
  st = check_layer(w_gate, "w_gate", act, !act);
  if (st != TPDQ_OK) return st;
  st = check_layer(w_up, "w_up", false, !act);
  if (st != TPDQ_OK) return st;
  st = check_layer(w_down, "w_down", act, !act);
  if (st != TPDQ_OK) return st;
  if (w_up->K != w_gate->K || w_up->N != w_gate->N || w_up->group_size != w_gate->group_size ||
      w_up->num_groups != w_gate->num_groups || w_up->layout != w_gate->layout ||
      w_up->ld_q != w_gate->ld_q || w_up->ld_s != w_gate->ld_s || w_up->ld_z != w_gate->ld_z ||
      w_up->zero_offset != w_gate->zero_offset)
    return fail(TPDQ_ERR_SHAPE,
                "w_up must match w_gate in shape, groups, layout, leading dimensions and zero offset");
  if (w_down->K != w_gate->N)
    return fail(TPDQ_ERR_SHAPE, "w_down->K=%d != w_gate->N=%d", w_down->K, w_gate->N);
  if (!X || !Y1 || !Y2_partial) return fail(TPDQ_ERR_NULL, "X, Y1 and Y2_partial are required");
  if (act && P1) return fail(TPDQ_ERR_SHAPE, "the act-order paths take no P1");
  if (!act && !P1) return fail(TPDQ_ERR_NULL, "the ordered path needs P1");
  if (ldx < w_gate->K) return fail(TPDQ_ERR_SHAPE, "ldx=%lld < K1=%d", (long long)ldx, w_gate->K);
  if (!aligned(X, 16) || ldx % 8)
    return fail(TPDQ_ERR_ALIGN, "X needs 16-byte alignment and ldx %% 8 == 0");
  if (!aligned(Y1, 16) || !aligned(Y2_partial, 8))
    return fail(TPDQ_ERR_ALIGN, "Y1 needs 16-byte and Y2_partial 8-byte alignment");
  const int meta = meta_mode(path);
  const size_t bound = tpdq_workspace_bytes(3, M, w_gate, w_down);
  const size_t need = std::max(gemm_ws_need(M, ldx, !act, w_gate, meta, dtype, true),
                               gemm_ws_need(M, w_gate->N, false, w_down, meta, dtype));
  if ((!act || need) && (!workspace || ws_bytes < bound))
    return fail(TPDQ_ERR_WORKSPACE, "gated MLP needs %zu workspace bytes, got %zu", bound, ws_bytes);
  if (workspace && !aligned(workspace, 16))
    return fail(TPDQ_ERR_ALIGN, "workspace needs 16-byte alignment");

  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  GemmIO io1, io2;
  io1.up = w_up;
  if (workspace && ws_bytes >= bound && mlp_prepared_y1(M, ldx, !act, w_gate, w_down, meta, dtype, true)) {
    io1.yp = (uint16_t*)(ws + gemm_ws_need(M, ldx, !act, w_gate, meta, dtype, true));
    io1.yp_natural = w_down->layout == TPDQ_LAYOUT_TILED ? 1 : 0;
    io2.x_prepared = true;
  }
  st = run_gemm((const uint16_t*)X, ldx, M, act ? nullptr : P1, w_gate, path, dtype, (uint16_t*)Y1,
                w_gate->N, ws, s, io1);
  if (st != TPDQ_OK) return st;
  if (io2.x_prepared)
    return run_gemm(io1.yp, w_gate->N, M, nullptr, w_down, path, dtype, (uint16_t*)Y2_partial,
                    w_down->N, ws, s, io2);
  return run_gemm((const uint16_t*)Y1, w_gate->N, M, nullptr, w_down, path, dtype,
                  (uint16_t*)Y2_partial, w_down->N, ws, s);
}

}  // extern "C"
