// C ABI of the MoARa optimizer library: validation, state, scheduling.
// Host code; every method step runs in the kernels of decompose.hip, gemm.hip
// and refresh.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/moara.h"
#include "common.h"
#include "gemm.h"
#include "refresh.h"


namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(MOARA_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr size_t ALIGN = 256;
size_t align_up(size_t x) { return (x + ALIGN - 1) & ~(ALIGN - 1); }

// ------------------------------------------------------------------ allocation-free scratch
// moara_step_noalloc takes every buffer beyond the caller's and the state's own memory
// (step and refresh descriptors, the refresh workspace) from this fixed array instead of
// allocating. Each GPU the library runs on holds one copy until the process ends. In host
// code `scratch` names a host-side stand-in: the device address of a GPU's copy comes
// from hipGetSymbolAddress with that GPU current (scratch_init, called when a state is
// created) and only that address is ever handed to kernels or copies.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)MOARA_NOALLOC_SCRATCH_BYTES;
constexpr size_t NOALLOC_REF_DESC_BYTES = (size_t)8 << 20;   // refresh descriptors of one chunk
constexpr int MAX_DEVICES = 64;
}  // namespace
static __device__ __align__(256) char scratch[NOALLOC_SCRATCH_BYTES];
namespace {
std::mutex g_scratch_mu;
char* g_scratch_ptr[MAX_DEVICES] = {};
hipEvent_t g_scratch_ev[MAX_DEVICES] = {};   // recorded at the end of every no-alloc call on the GPU
bool g_scratch_ev_valid[MAX_DEVICES] = {};

int scratch_init(int dev) {
  if (dev < 0 || dev >= MAX_DEVICES) return fail(MOARA_E_ARG, "device %d out of range for the scratch table", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev]) return MOARA_OK;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p) return fail(MOARA_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
  hipEvent_t ev = nullptr;
  const hipError_t e2 = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
  if (e2 != hipSuccess) return fail(MOARA_E_HIP, "scratch event: %s", hipGetErrorString(e2));
  g_scratch_ptr[dev] = (char*)p;
  g_scratch_ev[dev] = ev;
  return MOARA_OK;
}

struct MatHost {
  int64_t m = 0, n = 0, L = 0, s = 0;
  int32_t r = 0, side = 0, k = 0;
  int64_t t = 0;
  bool hasP = false;
  bool refreshed = false;   // the library's refresh has written this matrix's record
  float *inv = nullptr, *dM = nullptr, *mag1 = nullptr, *mag2 = nullptr;
  void *exp1 = nullptr, *exp2 = nullptr;   // Optimizer_V moments, L x r, fp32 or bf16 (moment_dtype)
  float* P32 = nullptr;
  void *N = nullptr, *Pop = nullptr, *Ptop = nullptr;
  bool vpath = false;    // the decomposition writes V in bf16 for the large-tile projection
  void* V = nullptr;     // L x s bf16 direction workspace, blocked layout (kp_index, K = s)
  bool kp = false;       // Ptop (K = s), Pop and N (K = r) in the blocked layout too
};

struct TimedLaunch {
  int kind;
  hipEvent_t a, b;
};

}  // namespace

struct moara_state {
  moara_config cfg;
  int n = 0;
  int device = 0;
  std::vector<MatHost> mats;
  char* block = nullptr;        // all persistent device memory
  size_t block_bytes = 0;
  int32_t* info_dev = nullptr;  // 4 ints per matrix: the last refresh's record (RefDev::info)
  // descriptor staging: pinned host ring + one device arena (stream ordered)
  static constexpr int NSLOT = 8;
  char* host_ring = nullptr;
  char* dev_arena = nullptr;
  size_t arena_bytes = 0;
  hipEvent_t slot_ev[NSLOT] = {};
  bool slot_used[NSLOT] = {};
  int slot = 0;
  // refresh workspace
  char* ref_ws = nullptr;
  size_t ref_ws_bytes = 0;
  char* ref_arena = nullptr;      // device descriptors of the refresh (separate arena)
  size_t ref_arena_bytes = 0;
  char* ref_host = nullptr;
  // cross-stream order: recorded on the caller's stream at the end of every call that
  // enqueues work on the state; the next call's stream waits on it first
  hipEvent_t order_ev = nullptr;
  bool order_valid = false;
  // inside moara_step_noalloc: dev_arena, ref_arena and ref_ws point into the scratch
  // array (NoallocView) and nothing may be allocated
  bool noalloc = false;
  // timing
  bool timing = false;
  std::vector<TimedLaunch> pending;
  std::vector<hipEvent_t> ev_pool;
  int64_t launches[MOARA_NUM_KERNELS] = {};
  double total_ms[MOARA_NUM_KERNELS] = {};
};

namespace {

int elem_bytes(int dtype) { return dtype == MOARA_BF16 ? 2 : 4; }

// bf16 <-> fp32 on the host for the state-access calls: widening is exact; narrowing
// rounds to nearest, ties to even, and keeps NaN a quiet NaN
float host_bf16_to_f32(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}
uint16_t host_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

int validate_config(const moara_config* c) {
  if (!c) return fail(MOARA_E_ARG, "config is NULL");
  if (c->block_size < 1) return fail(MOARA_E_ARG, "block_size must be >= 1 (got %d)", c->block_size);
  if (!(c->beta1 >= 0.f && c->beta1 < 1.f) || !(c->beta2 >= 0.f && c->beta2 < 1.f))
    return fail(MOARA_E_ARG, "betas must lie in [0, 1)");
  if (!(c->adam_eps > 0.f) || !isfinite(c->adam_eps)) return fail(MOARA_E_ARG, "adam_eps must be > 0");
  if (!(c->decomp_eps >= 0.f) || !isfinite(c->decomp_eps)) return fail(MOARA_E_ARG, "decomp_eps must be >= 0");
  if (!isfinite(c->scale)) return fail(MOARA_E_ARG, "scale must be finite");
  if (c->weight_decay != 0.f) return fail(MOARA_E_UNSUPPORTED, "weight_decay != 0 is not supported (the method uses none)");
  if (c->refresh_interval < 0) return fail(MOARA_E_ARG, "refresh_interval must be >= 0");
  if (c->bias_correction != 0 && c->bias_correction != 1) return fail(MOARA_E_ARG, "bias_correction must be 0 or 1");
  if (c->decompose != 0 && c->decompose != 1) return fail(MOARA_E_ARG, "decompose must be 0 or 1");
  if (c->weight_dtype != MOARA_F32 && c->weight_dtype != MOARA_BF16) return fail(MOARA_E_ARG, "bad weight_dtype");
  if (c->grad_dtype != MOARA_F32) return fail(MOARA_E_UNSUPPORTED, "only fp32 gradients are supported");
  if (c->operand_dtype != MOARA_F32 && c->operand_dtype != MOARA_BF16) return fail(MOARA_E_ARG, "bad operand_dtype");
  if (c->refresh_oversample < -1) return fail(MOARA_E_ARG, "refresh_oversample must be >= -1");
  if (c->refresh_iters < 1 || c->refresh_iters > 1000) return fail(MOARA_E_ARG, "refresh_iters must be in [1, 1000]");
  if (c->zero_grad_mode != 0 && c->zero_grad_mode != 1) return fail(MOARA_E_ARG, "bad zero_grad_mode");
  if (c->moment_dtype != MOARA_F32 && c->moment_dtype != MOARA_BF16) return fail(MOARA_E_ARG, "bad moment_dtype");
  return MOARA_OK;
}

int resolve(const moara_config* cfg, const moara_matrix_desc* d, int32_t* rank, int32_t* side) {
  if (!cfg || !d || !rank || !side) return fail(MOARA_E_ARG, "NULL argument");
  if (d->rows < 1 || d->cols < 1) return fail(MOARA_E_SHAPE, "matrix shape %lldx%lld", (long long)d->rows, (long long)d->cols);
  if (d->rows > (1LL << 31) - 1 || d->cols > (1LL << 31) - 1) return fail(MOARA_E_SHAPE, "matrix dimension too large");
  if (d->module < 0 || d->module >= MOARA_NUM_MODULES) return fail(MOARA_E_ARG, "module id %d out of range", d->module);
  if (d->side < MOARA_SIDE_AUTO || d->side > MOARA_SIDE_RIGHT) return fail(MOARA_E_ARG, "bad side %d", d->side);
  if (d->rank_override < 0) return fail(MOARA_E_RANK, "rank_override must be >= 0");
  if (d->reserved != 0) return fail(MOARA_E_ARG, "descriptor reserved field must be 0");
  const int32_t r = d->rank_override > 0 ? d->rank_override : cfg->rank_table[d->module];
  const int64_t mn = std::min(d->rows, d->cols);
  if (r < 1 || r > mn) return fail(MOARA_E_RANK, "rank %d outside [1, min(m,n)=%lld] for module %d", r, (long long)mn, d->module);
  int sd = d->side;
  if (sd == MOARA_SIDE_AUTO) sd = (d->rows <= d->cols) ? MOARA_SIDE_LEFT : MOARA_SIDE_RIGHT;
  *rank = r;
  *side = sd;
  return MOARA_OK;
}

struct Layout {
  int64_t s, L, k;
};
Layout layout_of(const moara_matrix_desc& d, int side, int B) {
  Layout l;
  l.s = side == MOARA_SIDE_LEFT ? d.rows : d.cols;
  l.L = side == MOARA_SIDE_LEFT ? d.cols : d.rows;
  l.k = (d.cols + B - 1) / B;
  return l;
}

int32_t subspace_width(const moara_config& c, int64_t s, int32_t r) {
  const int64_t p = c.refresh_oversample < 0 ? r : c.refresh_oversample;
  return (int32_t)std::min<int64_t>(s, r + p);
}

// Shapes for which the decomposition materialises V in bf16 and the projection runs
// on the large-tile bf16 GEMM (see decompose.hip / gemm_nt.hip for the limits).
bool vpath_shape_ok(const moara_config& c, int64_t m, int64_t n, int side, int32_t r) {
  if (c.operand_dtype != MOARA_BF16 || !c.decompose) return false;
  const int B = c.block_size;
  if (B < 4 || B > 256 || (B & (B - 1))) return false;
  if (n % 4 || r % 4) return false;
  const int64_t k = (n + B - 1) / B;
  if (2 * m * n > 0x7FFFFFFFLL) return false;
  if (side == MOARA_SIDE_LEFT) return k <= DEC_VT_MAX_K && m % 32 == 0;
  return k <= DEC_ROW_MAX_K && n % 32 == 0;
}

size_t mat_state_bytes(const moara_config& c, int64_t m, int64_t n, int side, int64_t s, int64_t L, int64_t k,
                       int32_t r) {
  const int ob = elem_bytes(c.operand_dtype);
  size_t b = 0;
  if (vpath_shape_ok(c, m, n, side, r)) b += align_up(2 * (size_t)m * n);   // V workspace
  b += align_up(4 * m * k) * 4;          // inv, dM, mag1, mag2
  b += align_up((size_t)elem_bytes(c.moment_dtype) * L * r) * 2;   // exp1, exp2
  b += align_up((size_t)ob * L * r);     // N
  b += align_up(4 * s * r);              // P32
  b += align_up((size_t)ob * s * r) * 2; // Pop, Ptop
  return b;
}

// bf: the matrix runs its early subspace iterations on the bf16 V (other orientation
// of V and bf16 copies of the iterates)
size_t mat_refresh_bytes(int64_t s, int64_t L, int32_t w, int32_t r, bool bf) {
  const int64_t wpad = (w + 63) / 64 * 64;
  size_t b = 0;
  b += align_up(4 * (size_t)s * r) + align_up(4 * (size_t)r * w);   // Pw, Bt
  if (bf) b += 5 * align_up(2 * (size_t)s * L) + 2 * align_up(2 * (size_t)w * s) + 3 * align_up(2 * (size_t)w * L);
  b += align_up(4 * s * w) * 2;            // Z, Z2
  b += align_up(4 * L * w) * 2;            // Y, Y2
  b += align_up(8 * (size_t)w * w) * 2;    // C, X
  b += align_up(8);                        // cmax
  b += align_up(4 * (size_t)w * w);        // Rinv
  b += align_up(8 * (size_t)wpad * w);     // Zc (R, column-major)
  b += align_up(4 * 64);                   // off
  b += 2 * align_up(4 * (size_t)(wpad / 32 - 1) * (wpad / 64)) + align_up(4 * (size_t)(wpad / 32));   // Jacobi records
  b += align_up(4 * wpad) + align_up(8 * wpad);
  b += align_up(8 * 64 * (size_t)s) + align_up(8 * 64 * (size_t)r) + align_up(8 * (size_t)s) + align_up(4 * (size_t)r);  // completion
  return b;
}

// ------------------------------------------------------------------ staging
struct Stager {
  moara_state* st;
  char* host = nullptr;
  size_t used = 0;
  size_t cap = 0;
  template <typename T>
  size_t push(const T* p, size_t count) {
    const size_t off = used;
    const size_t bytes = sizeof(T) * count;
    if (used + bytes > cap) return (size_t)-1;
    memcpy(host + used, p, bytes);
    used = align_up(used + bytes);
    return off;
  }
};

int begin_stage(moara_state* st, Stager& sg) {
  const int s = st->slot;
  if (st->slot_used[s]) HIP_TRY(hipEventSynchronize(st->slot_ev[s]));
  sg.st = st;
  sg.host = st->host_ring + (size_t)s * st->arena_bytes;
  sg.used = 0;
  sg.cap = st->arena_bytes;
  return MOARA_OK;
}

int end_stage(moara_state* st, Stager& sg, hipStream_t stream) {
  const int s = st->slot;
  if (sg.used) HIP_TRY(hipMemcpyAsync(st->dev_arena, sg.host, sg.used, hipMemcpyHostToDevice, stream));
  HIP_TRY(hipEventRecord(st->slot_ev[s], stream));
  st->slot_used[s] = true;
  st->slot = (s + 1) % moara_state::NSLOT;
  return MOARA_OK;
}

// ------------------------------------------------------------------ stream order
// Every call that enqueues work on a state makes its stream wait for the work the
// previous call enqueued (on whatever stream), and records the event again when it
// returns: calls on one state run in call order even across streams, so the shared
// descriptor arenas, workspaces and state tensors are never used by two streams at once.
// The state's memory and its GPU's scratch live on the device that was current when the
// state was created; a call enqueues on `stream`, which belongs to the current device.
static int check_device(const moara_state* st) {
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return fail(MOARA_E_HIP, "hipGetDevice failed");
  if (cur != st->device)
    return fail(MOARA_E_STATE, "the current HIP device is %d but the state lives on device %d", cur, st->device);
  return MOARA_OK;
}

struct StreamOrder {
  moara_state* st;
  hipStream_t stream;
  hipError_t err = hipSuccess;
  StreamOrder(moara_state* s, hipStream_t str) : st(s), stream(str) {
    if (st->order_valid) err = hipStreamWaitEvent(stream, st->order_ev, 0);
  }
  ~StreamOrder() {
    if (hipEventRecord(st->order_ev, stream) == hipSuccess) st->order_valid = true;
  }
};
#define ORDER_ON(st_, stream_)                                                               \
  if (const int dev_rc_ = check_device(st_)) return dev_rc_;                                \
  StreamOrder order_guard_((st_), (stream_));                                               \
  if (order_guard_.err != hipSuccess)                                                       \
    return fail(MOARA_E_HIP, "hipStreamWaitEvent: %s", hipGetErrorString(order_guard_.err))

// ------------------------------------------------------------------ timing
hipEvent_t get_event(moara_state* st) {
  if (!st->ev_pool.empty()) {
    hipEvent_t e = st->ev_pool.back();
    st->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct TimerScope {
  moara_state* st;
  int kind;
  hipStream_t stream;
  hipEvent_t a = nullptr;
  TimerScope(moara_state* s, int k, hipStream_t str) : st(s), kind(k), stream(str) {
    if (st->timing) {
      a = get_event(st);
      if (a && hipEventRecord(a, stream) != hipSuccess) {   // no bracket: this launch goes untimed
        st->ev_pool.push_back(a);
        a = nullptr;
      }
    }
  }
  ~TimerScope() {
    if (st->timing && a) {
      hipEvent_t b = get_event(st);
      if (b && hipEventRecord(b, stream) == hipSuccess) {
        st->pending.push_back({kind, a, b});
      } else {
        st->ev_pool.push_back(a);
        if (b) st->ev_pool.push_back(b);
      }
    }
  }
};

int collect_timing(moara_state* st, hipStream_t stream) {
  if (st->pending.empty()) return MOARA_OK;
  (void)stream;   // the events may sit on several streams: wait for each one itself
  for (auto& tl : st->pending) {
    float ms = 0.f;
    HIP_TRY(hipEventSynchronize(tl.b));
    HIP_TRY(hipEventElapsedTime(&ms, tl.a, tl.b));
    st->launches[tl.kind] += 1;
    st->total_ms[tl.kind] += ms;
    st->ev_pool.push_back(tl.a);
    st->ev_pool.push_back(tl.b);
  }
  st->pending.clear();
  return MOARA_OK;
}

// ------------------------------------------------------------------ step launch
int vec_flags_g(const float* G, int64_t n) { return (((uintptr_t)G & 15) == 0 && (n & 3) == 0) ? 1 : 0; }
int vec_flags_op(const void* p, int64_t ld, int operand_bf16) {
  const int64_t q = operand_bf16 ? 8 : 4;
  return (((uintptr_t)p & 15) == 0 && (ld % q) == 0) ? 1 : 0;
}

// Enable the buffer-load fast path (vec bit 2) when both operands allow 16-byte
// loads and every offset a tile can form (extent plus a 256-row overhang) fits
// in the 32-bit buffer offset.
void set_extents(GemmProb& g, size_t a_bytes, size_t a_row_bytes, size_t b_bytes, size_t b_row_bytes,
                 size_t inv_bytes, size_t inv_row_bytes) {
  const size_t lim = (size_t)0xFFFFFFFFu;
  const bool ok = a_bytes + 256 * a_row_bytes < lim && b_bytes + 256 * b_row_bytes < lim &&
                  inv_bytes + 256 * inv_row_bytes < lim;
  g.a_bytes = ok ? (uint32_t)a_bytes : 0u;
  g.b_bytes = ok ? (uint32_t)b_bytes : 0u;
  g.inv_bytes = ok ? (uint32_t)inv_bytes : 0u;
  if (ok && (g.vec & 3) == 3) g.vec |= 4;
}

StepParams make_params(const moara_state* st, float lr) {
  StepParams p{};
  p.B = st->cfg.block_size;
  p.decompose = st->cfg.decompose;
  p.weight_bf16 = st->cfg.weight_dtype == MOARA_BF16;
  p.beta1 = st->cfg.beta1;
  p.beta2 = st->cfg.beta2;
  p.adam_eps = st->cfg.adam_eps;
  p.decomp_eps = st->cfg.decomp_eps;
  p.lr = lr;
  p.scale = st->cfg.scale;
  return p;
}

GemmUniform make_uniform(const moara_state* st, float lr) {
  GemmUniform u{};
  u.B = st->cfg.block_size;
  u.weight_bf16 = st->cfg.weight_dtype == MOARA_BF16;
  u.moment_bf16 = st->cfg.moment_dtype == MOARA_BF16;
  u.beta1 = st->cfg.beta1;
  u.beta2 = st->cfg.beta2;
  u.adam_eps = st->cfg.adam_eps;
  u.lr = lr;
  u.scale = st->cfg.scale;
  return u;
}

// Decompose (inv, and optionally Optimizer_M) for the listed matrices.
// usev (indexed by matrix, may be null): write the bf16 V for that matrix as well.
int run_decompose(moara_state* st, const std::vector<int>& idx, const void* const* grads, bool adam_m,
                  hipStream_t stream, const std::vector<char>* usev = nullptr) {
  if (idx.empty()) return MOARA_OK;
  std::vector<MatDev> md, mvt;
  uint32_t tiles = 0, tiles_vt = 0;
  for (int i : idx) {
    const MatHost& h = st->mats[i];
    MatDev d{};
    d.G = (const float*)grads[i];
    d.m = h.m; d.n = h.n; d.k = h.k; d.r = h.r; d.side = h.side;
    d.inv = h.inv; d.dM = h.dM; d.mag1 = h.mag1; d.mag2 = h.mag2;
    const double t1 = (double)(h.t + 1);
    d.bc1 = st->cfg.bias_correction ? (float)(1.0 - pow((double)st->cfg.beta1, t1)) : 1.f;
    d.bc2 = st->cfg.bias_correction ? (float)(1.0 - pow((double)st->cfg.beta2, t1)) : 1.f;
    const bool wv = usev && (*usev)[i];
    if (wv && h.side == MOARA_SIDE_LEFT) {
      d.Vb = (bf16*)h.V; d.vt = 1;
      d.tile_dec = tiles_vt;
      tiles_vt += (uint32_t)decompose_vt_tiles(h.m);
      mvt.push_back(d);
    } else {
      d.Vb = wv ? (bf16*)h.V : nullptr; d.vt = 0;
      d.tile_dec = tiles;
      tiles += (uint32_t)decompose_tiles(h.m);
      md.push_back(d);
    }
  }
  Stager sg;
  int rc = begin_stage(st, sg);
  if (rc) return rc;
  const size_t off = md.empty() ? 0 : sg.push(md.data(), md.size());
  const size_t offv = mvt.empty() ? 0 : sg.push(mvt.data(), mvt.size());
  if (off == (size_t)-1 || offv == (size_t)-1) return fail(MOARA_E_OOM, "descriptor arena too small");
  rc = end_stage(st, sg, stream);
  if (rc) return rc;
  TimerScope ts(st, MOARA_KERN_DECOMPOSE, stream);
  if (!mvt.empty()) {
    StepParams p = make_params(st, 0.f);
    p.nmat = (int)mvt.size();
    p.total_dec = tiles_vt;
    HIP_TRY(launch_decompose_vt((const MatDev*)(st->dev_arena + offv), p, adam_m ? 1 : 0, stream));
  }
  if (!md.empty()) {
    StepParams p = make_params(st, 0.f);
    p.nmat = (int)md.size();
    p.total_dec = tiles;
    const MatDev* dev = (const MatDev*)(st->dev_arena + off);
    HIP_TRY(adam_m ? launch_decompose(dev, p, stream) : launch_decompose_inv_only(dev, p, stream));
  }
  return MOARA_OK;
}

// back_only (indexed by matrix, may be null): N was formed without a projection (zero
// gradient); only the back-projection and update run for that matrix.
int run_project_back(moara_state* st, const std::vector<int>& idx, void* const* weights, const void* const* grads,
                     float lr, hipStream_t stream, const std::vector<char>* usev = nullptr,
                     const std::vector<char>* back_only = nullptr) {
  const int ob = st->cfg.operand_dtype == MOARA_BF16;
  const int kind = ob ? KIND_BF16 : KIND_F32;
  const int wbf = st->cfg.weight_dtype == MOARA_BF16;
  std::vector<GemmProb> left, right, back, pnt, bnt;
  uint32_t tl = 0, tr = 0, tb = 0, tpn = 0, tbn = 0;
  for (int i : idx) {
    const MatHost& h = st->mats[i];
    const double t1 = (double)(h.t + 1);
    const float bc1 = st->cfg.bias_correction ? (float)(1.0 - pow((double)st->cfg.beta1, t1)) : 1.f;
    const float bc2 = st->cfg.bias_correction ? (float)(1.0 - pow((double)st->cfg.beta2, t1)) : 1.f;
    bool proj_done = false;
    if (usev && (*usev)[i] &&
        gemm_nt_eligible(EP_ADAM, h.L, h.r, h.s, h.s, h.s, h.r, h.V, h.Ptop, h.N, wbf)) {
      // V was written by this step's decomposition: R^(T) (L x r) = V' (L x s) * Ptop^T
      GemmProb g{};
      g.M = h.L; g.N = h.r; g.K = h.s;
      g.a = h.V; g.lda = h.s;
      g.b = h.Ptop; g.ldb = h.s;
      g.c = h.N; g.ldc = h.r;
      g.kp = 1 | (h.kp ? 2 | 4 : 0);
      g.e1 = (float*)h.exp1; g.e2 = (float*)h.exp2;
      g.bc1 = bc1; g.bc2 = bc2;
      g.a_bytes = (uint32_t)(2 * (size_t)h.L * h.s);
      g.b_bytes = (uint32_t)(2 * (size_t)h.r * h.s);
      g.tiles_n = gemm_nt_tiles_n(g.N);
      g.tile_start = tpn;
      tpn += gemm_nt_tiles_m(g.M) * g.tiles_n;
      pnt.push_back(g);
      proj_done = true;
    }
    {
      const size_t rows_a = h.side == MOARA_SIDE_LEFT ? h.s : h.L, rows_b = h.side == MOARA_SIDE_LEFT ? h.L : h.s;
      const void* ba = h.side == MOARA_SIDE_LEFT ? h.Pop : h.N;
      const void* bb = h.side == MOARA_SIDE_LEFT ? h.N : h.Pop;
      if (ob && gemm_nt_eligible(EP_UPDATE, h.m, h.n, h.r, h.r, h.r, h.n, ba, bb, weights[i], wbf)) {
        GemmProb b{};
        b.M = h.m; b.N = h.n; b.K = h.r;
        b.a = ba; b.b = bb;
        b.lda = h.r; b.ldb = h.r;
        b.kp = h.kp ? 3 : 0;
        b.c = weights[i]; b.ldc = h.n;
        b.dM = st->cfg.decompose ? h.dM : nullptr; b.dM_ld = h.k;
        b.a_bytes = (uint32_t)(2 * rows_a * h.r);
        b.b_bytes = (uint32_t)(2 * rows_b * h.r);
        b.tiles_n = gemm_nt_tiles_n(b.N);
        b.tile_start = tbn;
        tbn += gemm_nt_tiles_m(b.M) * b.tiles_n;
        bnt.push_back(b);
      } else {
        GemmProb b{};
        b.M = h.m; b.N = h.n; b.K = h.r;
        b.a = ba; b.b = bb;
        b.lda = h.r; b.ldb = h.r;
        b.kp = h.kp ? 3 : 0;
        b.c = weights[i]; b.ldc = h.n;
        b.dM = st->cfg.decompose ? h.dM : nullptr; b.dM_ld = h.k;
        b.tiles_n = gemm_tiles_n(kind, b.N);
        b.vec = vec_flags_op(b.a, h.r, ob) | (vec_flags_op(b.b, h.r, ob) << 1);
        const size_t e = ob ? 2 : 4;
        set_extents(b, e * rows_a * h.r, e * h.r, e * rows_b * h.r, e * h.r, 0, 0);
        b.tile_start = tb;
        tb += gemm_tiles_m(kind, b.M) * b.tiles_n;
        back.push_back(b);
      }
    }
    if (proj_done || (back_only && (*back_only)[i])) continue;
    GemmProb g{};
    g.M = h.L; g.N = h.r; g.K = h.s;
    g.a = grads[i]; g.lda = h.n;
    g.inv = st->cfg.decompose ? h.inv : nullptr; g.inv_ld = h.k;
    g.b = h.Ptop; g.ldb = h.s;
    g.c = h.N; g.ldc = h.r;
    g.kp = h.kp ? 2 | 4 : 0;
    g.e1 = (float*)h.exp1; g.e2 = (float*)h.exp2;
    g.bc1 = bc1;
    g.bc2 = bc2;
    g.tiles_n = gemm_tiles_n(kind, g.N);
    g.vec = vec_flags_g((const float*)grads[i], h.n) | (vec_flags_op(h.Ptop, h.s, ob) << 1);
    set_extents(g, 4 * (size_t)h.m * h.n, 4 * (size_t)h.n, (size_t)(ob ? 2 : 4) * h.r * h.s, (size_t)(ob ? 2 : 4) * h.s,
                g.inv ? 4 * (size_t)h.m * h.k : 0, 4 * (size_t)h.k);
    const uint32_t nt = gemm_tiles_m(kind, g.M) * g.tiles_n;
    if (h.side == MOARA_SIDE_LEFT) { g.tile_start = tl; tl += nt; left.push_back(g); }
    else { g.tile_start = tr; tr += nt; right.push_back(g); }
  }
  Stager sg;
  int rc = begin_stage(st, sg);
  if (rc) return rc;
  const size_t ol = left.empty() ? 0 : sg.push(left.data(), left.size());
  const size_t orr = right.empty() ? 0 : sg.push(right.data(), right.size());
  const size_t obk = back.empty() ? 0 : sg.push(back.data(), back.size());
  const size_t opn = pnt.empty() ? 0 : sg.push(pnt.data(), pnt.size());
  const size_t obn = bnt.empty() ? 0 : sg.push(bnt.data(), bnt.size());
  if (ol == (size_t)-1 || orr == (size_t)-1 || obk == (size_t)-1 || opn == (size_t)-1 || obn == (size_t)-1)
    return fail(MOARA_E_OOM, "descriptor arena too small");
  rc = end_stage(st, sg, stream);
  if (rc) return rc;
  const GemmUniform u = make_uniform(st, lr);
  {
    TimerScope ts(st, MOARA_KERN_PROJECT, stream);
    if (!pnt.empty())
      HIP_TRY(launch_gemm_nt(EP_ADAM, (const GemmProb*)(st->dev_arena + opn), (int)pnt.size(), tpn, u, stream));
    if (!right.empty())
      HIP_TRY(launch_gemm(kind, A_G_ROW, B_KC, EP_ADAM, (const GemmProb*)(st->dev_arena + orr), (int)right.size(), tr, u, stream));
    if (!left.empty())
      HIP_TRY(launch_gemm(kind, A_G_TRANS, B_KC, EP_ADAM, (const GemmProb*)(st->dev_arena + ol), (int)left.size(), tl, u, stream));
  }
  {
    TimerScope ts(st, MOARA_KERN_BACKPROJ, stream);
    if (!bnt.empty())
      HIP_TRY(launch_gemm_nt(EP_UPDATE, (const GemmProb*)(st->dev_arena + obn), (int)bnt.size(), tbn, u, stream));
    if (!back.empty())
      HIP_TRY(launch_gemm(kind, A_KC, B_KC, EP_UPDATE, (const GemmProb*)(st->dev_arena + obk), (int)back.size(), tb, u, stream));
  }
  return MOARA_OK;
}

// Zero-gradient step (zero_grad_mode 1) for the listed matrices: a refresh that falls due
// keeps the projector (V = 0), or sets the canonical one if there is none; then
// Optimizer_M and Optimizer_V on zero inputs (k_zero_grad). The back-projection and the
// update follow in run_project_back.
int run_zero_grad(moara_state* st, const std::vector<int>& zidx, hipStream_t stream) {
  if (zidx.empty()) return MOARA_OK;
  const int T = st->cfg.refresh_interval;
  const int obf = st->cfg.operand_dtype == MOARA_BF16;
  for (int i : zidx) {
    MatHost& h = st->mats[i];
    if (T > 0 && h.t % T == 0 && !h.hasP) {
      HIP_TRY(launch_canonical_projector(h.P32, h.Pop, h.Ptop, h.s, h.r, obf, h.kp ? 1 : 0, stream));
      h.hasP = true;
    }
  }
  std::vector<MatDev> md;
  uint32_t tiles = 0;
  for (int i : zidx) {
    const MatHost& h = st->mats[i];
    MatDev d{};
    d.m = h.m; d.n = h.n; d.k = h.k; d.r = h.r; d.side = h.side; d.L = (int32_t)h.L; d.s = (int32_t)h.s;
    d.dM = h.dM; d.mag1 = h.mag1; d.mag2 = h.mag2;
    d.exp1 = (float*)h.exp1; d.exp2 = (float*)h.exp2; d.N = h.N;
    d.mom_bf16 = st->cfg.moment_dtype == MOARA_BF16;
    d.n_bf16 = obf; d.n_kp = h.kp ? 1 : 0;
    const double t1 = (double)(h.t + 1);
    d.bc1 = st->cfg.bias_correction ? (float)(1.0 - pow((double)st->cfg.beta1, t1)) : 1.f;
    d.bc2 = st->cfg.bias_correction ? (float)(1.0 - pow((double)st->cfg.beta2, t1)) : 1.f;
    d.tile_dec = tiles;
    tiles += zero_grad_tiles(st->cfg.decompose ? h.m * h.k : 0, h.L * h.r);
    md.push_back(d);
  }
  Stager sg;
  int rc = begin_stage(st, sg);
  if (rc) return rc;
  const size_t off = sg.push(md.data(), md.size());
  if (off == (size_t)-1) return fail(MOARA_E_OOM, "descriptor arena too small");
  if ((rc = end_stage(st, sg, stream))) return rc;
  StepParams p = make_params(st, 0.f);
  p.nmat = (int)md.size();
  p.total_dec = tiles;
  TimerScope ts(st, MOARA_KERN_DECOMPOSE, stream);
  HIP_TRY(launch_zero_grad((const MatDev*)(st->dev_arena + off), p, stream));
  return MOARA_OK;
}

// ------------------------------------------------------------------ refresh driver
struct RefMat {
  int idx;
  bool bf;               // iterations on the bf16 V (large-tile GEMMs; the last ones split)
  void *XL, *Zt, *Yt;    // bf16: V as s x L; iterates Z^T (w x s) and Y^T (w x L)
  void *VKm, *VKl, *XLm, *XLl;   // split products: V's further bf16 parts (as L x s and s x L) ...
  void *Ztlo, *Ytlo, *Ytl2;      // ... and the iterates' bf16 parts (Y^T in three for the last product)
  float *Pw, *Bt;        // Ritz vectors before signs (s x r), (R J)_top^T (r x w)
  int64_t s, L;
  int32_t w, wpad;
  float *Z, *Z2, *Y, *Y2, *Rinv;
  double *C, *X, *cmax, *Zc, *norms;
  uint32_t* off;
  int32_t* order;
  uint32_t *jconv, *jmod;   // Jacobi pair and block records
  float* jmx;
  // bf16 path, early orthonormalisations: the parts of Z2 (three s x w bf16 arrays, blocked,
  // K = w) and of R^{-1} transposed (three w x w, blocked): they live in Y..Y2 and in X,
  // which hold nothing between the first and the last iteration (Y, Y2: last iteration
  // only; X: read inside the factorisation only)
  void *Z2p, *Rtp;
  double* cw;            // basis completion workspace (s x 64, r x 64, s)
  int32_t* sidx;         // basis completion indices (r)
};

int ensure_ref_ws(moara_state* st, size_t bytes) {
  if (bytes <= st->ref_ws_bytes) return MOARA_OK;
  if (st->noalloc)
    return fail(MOARA_E_UNSUPPORTED, "refresh workspace of %zu bytes exceeds the no-alloc scratch (%zu bytes)", bytes,
                st->ref_ws_bytes);
  if (st->ref_ws) {
    HIP_TRY(hipDeviceSynchronize());
    (void)hipFree(st->ref_ws);
    st->ref_ws = nullptr;
    st->ref_ws_bytes = 0;
  }
  if (hipMalloc(&st->ref_ws, bytes) != hipSuccess) {
    st->ref_ws = nullptr;
    return fail(MOARA_E_OOM, "refresh workspace of %zu bytes", bytes);
  }
  st->ref_ws_bytes = bytes;
  return MOARA_OK;
}

constexpr int MAX_SWEEPS = 14;

// One refresh pass over a chunk of matrices. Buffer roles are fixed:
//   Z <- Gaussian (used as it is when w <= s / 2 for every matrix of the state: such a
//        block has condition number below 6, and orthonormalising it would not change
//        the subspace the iteration sees; wider blocks go through Z2 <- Gaussian,
//        Z <- orth(Z2) first)
//   repeat: Y <- X Z ; Z2 <- X^T Y ; Z <- orth(Z2)        (q - 1 times)
//   last  : Y <- X Z ; Y2 <- orth(Y) ; Z2 <- X^T Y2 ; Jacobi on Z2 ; P <- top r
// usev (indexed by matrix, may be null): the bf16 V of that matrix was written by this
// step's decomposition, so its early subspace iterations can run on bf16 MFMA.
// The last iterations run at fp32 accuracy: fp32 products on G and inv, or, for matrices
// with a bf16 V, split bf16 products (operand + residual, three MFMA products per GEMM).
constexpr int REFRESH_F32_ITERS = 3;
// of which the last ones use the five-product split (the others three products)
#ifndef MOARA_SPLIT5_ITERS
#define MOARA_SPLIT5_ITERS 2
#endif
constexpr int REFRESH_SPLIT5_ITERS = MOARA_SPLIT5_ITERS;

int refresh_chunk(moara_state* st, const std::vector<int>& idx, const void* const* grads, hipStream_t stream,
                  const std::vector<char>* usev) {
  const moara_config& c = st->cfg;
  size_t need = 0;
  std::vector<RefMat> rm;
  for (int i : idx) {
    const MatHost& h = st->mats[i];
    RefMat x{};
    x.idx = i; x.s = h.s; x.L = h.L;
    x.w = subspace_width(c, h.s, h.r);
    x.wpad = (x.w + 63) / 64 * 64;
    x.bf = usev && (*usev)[i] && c.refresh_iters > REFRESH_F32_ITERS && x.w % 8 == 0 &&
           gemm_nt_eligible(EP_STORE_BF16, x.w, h.L, h.s, h.s, h.s, h.L, h.V, h.V, h.V, 0) &&
           gemm_nt_eligible(EP_STORE, h.s, x.w, h.L, h.L, h.L, x.w, h.V, h.V, h.V, 0) &&
           gemm_nt_eligible(EP_STORE, h.L, x.w, h.s, h.s, h.s, x.w, h.V, h.V, h.V, 0);
    need += mat_refresh_bytes(h.s, h.L, x.w, h.r, x.bf);
    rm.push_back(x);
  }
  int rc = ensure_ref_ws(st, need);
  if (rc) return rc;
  char* p = st->ref_ws;
  auto take = [&](size_t b) { char* q = p; p += align_up(b); return q; };
  auto h_r_of = [&](const RefMat& x) { return (size_t)st->mats[x.idx].r; };
  for (auto& x : rm) {
    if (x.bf) {
      x.XL = take(2 * (size_t)x.s * x.L);
      x.Zt = take(2 * (size_t)x.w * x.s);
      x.Yt = take(2 * (size_t)x.w * x.L);
      x.VKm = take(2 * (size_t)x.s * x.L);
      x.VKl = take(2 * (size_t)x.s * x.L);
      x.XLm = take(2 * (size_t)x.s * x.L);
      x.XLl = take(2 * (size_t)x.s * x.L);
      x.Ztlo = take(2 * (size_t)x.w * x.s);
      x.Ytlo = take(2 * (size_t)x.w * x.L);
      x.Ytl2 = take(2 * (size_t)x.w * x.L);
    }
    x.Z = (float*)take(4 * x.s * x.w);
    x.Z2 = (float*)take(4 * x.s * x.w);
    x.Y = (float*)take(4 * x.L * x.w);
    x.Y2 = (float*)take(4 * x.L * x.w);
    x.C = (double*)take(8 * (size_t)x.w * x.w);
    x.X = (double*)take(8 * (size_t)x.w * x.w);
    x.cmax = (double*)take(8);
    x.Rinv = (float*)take(4 * (size_t)x.w * x.w);
    x.Zc = (double*)take(8 * (size_t)x.wpad * x.w);
    x.Pw = (float*)take(4 * (size_t)x.s * h_r_of(x));
    x.Bt = (float*)take(4 * (size_t)h_r_of(x) * x.w);
    x.off = (uint32_t*)take(4 * 64);
    {
      const size_t nbj = (size_t)x.wpad / JB, npr = (nbj - 1) * (nbj / 2);
      x.jconv = (uint32_t*)take(4 * npr);
      x.jmx = (float*)take(4 * npr);
      x.jmod = (uint32_t*)take(4 * nbj);
    }
    x.order = (int32_t*)take(4 * x.wpad);
    x.norms = (double*)take(8 * x.wpad);
    x.cw = (double*)take(8 * 64 * (size_t)x.s + 8 * 64 * h_r_of(x) + 8 * (size_t)x.s);
    x.sidx = (int32_t*)take(4 * h_r_of(x));
    x.Z2p = x.Y;    // 6 s w bytes <= the 8 L w of Y and Y2 (taken one after the other) when 3 s <= 4 L
    x.Rtp = x.X;    // 6 w^2 bytes <= 8 w^2
  }
  const int nm = (int)rm.size();
  const int kind = KIND_F32;
  const GemmUniform u = make_uniform(st, 0.f);

  // the Gaussian start is orthonormalised only if some block of the state is wider than
  // s / 2 (decided over the whole state, so a matrix's refresh does not depend on how the
  // matrices are split into chunks or which of them are active)
  bool orth0 = false;
  for (int i = 0; i < st->n; ++i) {
    const MatHost& h = st->mats[i];
    orth0 = orth0 || 2 * (int64_t)subspace_width(c, h.s, h.r) > h.s;
  }
  std::vector<RefDev> rd(nm);
  uint32_t tg = 0, tj = 0, tc = 0, tnorm = 0;
  int nb_max = 2;
  for (int q = 0; q < nm; ++q) {
    const RefMat& x = rm[q];
    const MatHost& h = st->mats[x.idx];
    RefDev& d = rd[q];
    d.s = x.s; d.L = x.L; d.w = x.w; d.wpad = x.wpad; d.r = h.r;
    d.operand_bf16 = c.operand_dtype == MOARA_BF16;
    d.seed = c.refresh_seed * 0x9E3779B97F4A7C15ull + (uint64_t)(x.idx + 1) * 0xD1B54A32D192ED03ull;
    d.Z = x.Z2; d.Z0 = orth0 ? x.Z2 : x.Z; d.C = x.C; d.X = x.X; d.cmax = x.cmax; d.Rinv = x.Rinv; d.Zc = x.Zc;
    d.jl = x.w; d.Q = x.Z; d.Pw = x.Pw; d.Bt = x.Bt;
    d.P32 = h.P32; d.Pop = h.Pop; d.Ptop = h.Ptop; d.kp = h.kp ? 1 : 0;
    d.off = x.off; d.order = x.order; d.norms = x.norms;
    d.jconv = x.jconv; d.jmx = x.jmx; d.jmod = x.jmod;
    d.tile_gauss = tg; tg += gauss_tiles(x.s, x.w);
    d.tile_jac = tj; tj += jacobi_tiles(x.wpad);
    d.tile_cm = tc; tc += r_colmajor_tiles(x.w, x.wpad);
    d.tile_norm = tnorm; tnorm += norm_tiles(x.wpad);
    d.has_prev = h.hasP ? 1 : 0;
    d.max_sweeps = MAX_SWEEPS;
    d.info = st->info_dev + 4 * (size_t)x.idx;
    d.cw = x.cw;
    d.sidx = x.sidx;
    nb_max = std::max(nb_max, x.wpad / JB);
  }
  auto gram_list = [&](bool onY) {
    std::vector<GramProb> g(nm);
    uint32_t t = 0;
    for (int q = 0; q < nm; ++q) {
      const RefMat& x = rm[q];
      GramProb& gp = g[q];
      gp.A = onY ? x.Y : x.Z2;
      gp.rows = onY ? x.L : x.s;
      gp.lda = x.w; gp.C = x.C; gp.w = x.w;
      gp.tiles = (x.w + 63) / 64;
      gp.tile_start = t;
      t += gram_tiles(x.w);
    }
    return std::make_pair(g, t);
  };
  auto apply_list = [&](bool onY, bool only_f32 = false) {   // Z = Z2 Rinv  or  Y2 = Y Rinv
    std::vector<GemmProb> g;
    uint32_t t = 0;
    for (int q = 0; q < nm; ++q) {
      const RefMat& x = rm[q];
      if (only_f32 && x.bf) continue;
      g.emplace_back();
      GemmProb& gp = g.back();
      gp.M = onY ? x.L : x.s; gp.N = x.w; gp.K = x.w;
      gp.a = onY ? (const void*)x.Y : (const void*)x.Z2;
      gp.lda = x.w;
      gp.b = x.Rinv; gp.ldb = x.w;
      gp.tri_b = 1;   // Rinv is upper triangular (its lower part is zero)
      gp.c = onY ? (void*)x.Y2 : (void*)x.Z;
      gp.ldc = x.w;
      gp.tiles_n = gemm_tiles_n(kind, gp.N);
      gp.vec = vec_flags_op(gp.a, x.w, 0) | (vec_flags_op(gp.b, x.w, 0) << 1);
      set_extents(gp, 4 * (size_t)gp.M * x.w, 4 * (size_t)x.w, 4 * (size_t)x.w * x.w, 4 * (size_t)x.w, 0, 0);
      gp.tile_start = t;
      t += gemm_tiles_m(kind, gp.M) * gp.tiles_n;
    }
    return std::make_pair(g, t);
  };
  // Y = X Z  (tall: M = L, K = s)   or   Z2 = X^T Yin  (M = s, K = L)
  auto big_list = [&](int side, bool xt, bool fromY2, bool only_f32 = false) {
    std::vector<GemmProb> g;
    uint32_t t = 0;
    for (int q = 0; q < nm; ++q) {
      const RefMat& x = rm[q];
      const MatHost& h = st->mats[x.idx];
      if (h.side != side || (only_f32 && x.bf)) continue;
      GemmProb gp{};
      gp.M = xt ? x.s : x.L; gp.N = x.w; gp.K = xt ? x.L : x.s;
      gp.a = grads[x.idx]; gp.lda = h.n;
      gp.inv = c.decompose ? h.inv : nullptr; gp.inv_ld = h.k;
      gp.b = xt ? (fromY2 ? x.Y2 : x.Y) : x.Z; gp.ldb = x.w;
      gp.c = xt ? x.Z2 : x.Y; gp.ldc = x.w;
      gp.tiles_n = gemm_tiles_n(kind, gp.N);
      gp.vec = vec_flags_g((const float*)grads[x.idx], h.n) | (vec_flags_op(gp.b, x.w, 0) << 1);
      set_extents(gp, 4 * (size_t)h.m * h.n, 4 * (size_t)h.n, 4 * (size_t)gp.K * x.w, 4 * (size_t)x.w,
                  gp.inv ? 4 * (size_t)h.m * h.k : 0, 4 * (size_t)h.k);
      gp.tile_start = t;
      t += gemm_tiles_m(kind, gp.M) * gp.tiles_n;
      g.push_back(gp);
    }
    return std::make_pair(g, t);
  };
  // workgroup prefixes of the blocked Cholesky / inverse launches (same for every orth of the chunk)
  int nbmax = 1;
  for (auto& x : rm) nbmax = std::max(nbmax, chol_blocks(x.w));
  const int nlev = trtri_levels(nbmax);
  std::vector<uint32_t> pan_pref((size_t)nbmax * nm), upd_pref((size_t)nbmax * nm), inv_pref((size_t)std::max(1, nlev) * nm);
  std::vector<uint32_t> pan_tot(nbmax), upd_tot(nbmax), inv_tot(std::max(1, nlev));
  for (int k = 0; k < nbmax; ++k) {
    uint32_t tp = 0, tu = 0;
    for (int q = 0; q < nm; ++q) {
      const int nb = chol_blocks(rm[q].w);
      const int T = std::max(0, nb - k - 1);
      pan_pref[(size_t)k * nm + q] = tp; tp += (uint32_t)T;
      // row(k), k >= 1: one workgroup per matrix for the diagonal block (numbered first),
      // then the blocks c = k+1 .. nb-1 by prefix
      upd_pref[(size_t)k * nm + q] = tu; tu += (uint32_t)(k >= 1 && k < nb ? nb - k - 1 : 0);
    }
    pan_tot[k] = tp; upd_tot[k] = k >= 1 ? (uint32_t)nm + tu : 0;
  }
  for (int l = 1; l <= nlev; ++l) {   // recursive-doubling levels of the triangular inverse
    uint32_t ti = 0;
    for (int q = 0; q < nm; ++q) {
      inv_pref[(size_t)(l - 1) * nm + q] = ti;
      ti += trtri_tiles(rm[q].w, l);
    }
    inv_tot[l - 1] = ti;
  }
  auto gZ2 = gram_list(false), gY = gram_list(true);
  auto aZ = apply_list(false), aY = apply_list(true), aZf = apply_list(false, true);
  // fp32 products on G and inv: the matrices without a bf16 V (every iteration) ...
  auto xzR = big_list(MOARA_SIDE_RIGHT, false, false, true), xzL = big_list(MOARA_SIDE_LEFT, false, false, true);
  auto xtR = big_list(MOARA_SIDE_RIGHT, true, false, true), xtL = big_list(MOARA_SIDE_LEFT, true, false, true);
  auto xt2R = big_list(MOARA_SIDE_RIGHT, true, true, true), xt2L = big_list(MOARA_SIDE_LEFT, true, true, true);
  // ... and, for the others, Z^T (bf16) = transpose(Z), Y^T = Z^T X_K^T, Z2 = X_L Y  (X_K: L x s = the
  // step's V workspace, X_L: s x L = its transpose); in the last REFRESH_F32_ITERS iterations
  // every operand is split into bf16 + bf16 residual (three products per GEMM, near fp32)
  // Ritz vectors: Pw = Q Bt^T (M = s, N = r, K = w)
  std::vector<GemmProb> pwl;
  uint32_t tpw = 0;
  for (int q = 0; q < nm; ++q) {
    const RefMat& x = rm[q];
    const int r = st->mats[x.idx].r;
    GemmProb gp{};
    gp.M = x.s; gp.N = r; gp.K = x.w;
    gp.a = x.Z; gp.lda = x.w; gp.b = x.Bt; gp.ldb = x.w; gp.c = x.Pw; gp.ldc = r;
    gp.tiles_n = gemm_tiles_n(kind, gp.N);
    gp.vec = vec_flags_op(gp.a, x.w, 0) | (vec_flags_op(gp.b, x.w, 0) << 1);
    set_extents(gp, 4 * (size_t)x.s * x.w, 4 * (size_t)x.w, 4 * (size_t)r * x.w, 4 * (size_t)x.w, 0, 0);
    gp.tile_start = tpw;
    tpw += gemm_tiles_m(kind, gp.M) * gp.tiles_n;
    pwl.push_back(gp);
  }
  std::vector<TransProb> tZ, tX, tZs, tY2, tR;
  std::vector<GemmProb> nY, nZ, nYs, nZs, nYf, nYs3, nZs3, nZf, qZ, qZs;
  std::vector<SplitProb> vlo;
  uint32_t ttz = 0, ttx = 0, tny = 0, tnz = 0, tvlo = 0, tnyf = 0, tty2 = 0, ttr = 0, tqz = 0;
  // The early orthonormalisations of the bf16-path matrices form the next iterate's bf16
  // copy Z^T (w x s, blocked) straight from split bf16 products, Z^T = (R^{-1})^T Z2^T with
  // both factors in three parts (about fp32 accuracy, as the fp32 GEMM it replaces), instead
  // of an fp32 GEMM followed by a transpose. Needs K = w in 32-steps for every such matrix.
  bool use_qz = false;
  for (const RefMat& x : rm) {
    if (!x.bf) continue;
    const MatHost& h = st->mats[x.idx];
    // (Z2's parts live in Y..Y2: 3 s <= 4 L, which the automatic side choice, s <= L, meets)
    use_qz = x.w % 32 == 0 && 3 * x.s <= 4 * x.L &&
             gemm_nt_eligible(EP_STORE_BF16, x.w, h.s, x.w, x.w, x.w, h.s, h.V, h.V, h.V, 0);
    if (!use_qz) break;
  }
  for (int q = 0; q < nm; ++q) {
    const RefMat& x = rm[q];
    if (!x.bf) continue;
    const MatHost& h = st->mats[x.idx];
    TransProb a{};
    a.in = x.Z; a.out = x.Zt; a.rows = x.s; a.cols = x.w; a.ldi = x.w; a.ldo = x.s; a.in_f32 = 1; a.out_kp = 1;
    a.tiles_c = (int32_t)((x.w + 63) / 64); a.tile_start = ttz; ttz += transpose_tiles(x.s, x.w);
    tZ.push_back(a);
    TransProb b{};
    b.in = h.V; b.out = x.XL; b.rows = x.L; b.cols = x.s; b.ldi = x.s; b.ldo = x.L; b.in_f32 = 0; b.in_kp = 1;
    b.out_kp = 1;
    b.tiles_c = (int32_t)((x.s + 63) / 64); b.tile_start = ttx; ttx += transpose_tiles(x.L, x.s);
    tX.push_back(b);
    GemmProb y{};
    y.M = x.w; y.N = x.L; y.K = x.s;
    y.a = x.Zt; y.lda = x.s; y.b = h.V; y.ldb = x.s; y.c = x.Yt; y.ldc = x.L;
    y.kp = 1 | 2 | 4;   // Zt, V and the output Yt in the blocked layout (K = s for Zt and V, L for Yt)
    y.a_bytes = (uint32_t)(2 * (size_t)x.w * x.s); y.b_bytes = (uint32_t)(2 * (size_t)x.L * x.s);
    y.tiles_n = gemm_nt_tiles_n(y.N); y.tile_start = tny; tny += gemm_nt_tiles_m(y.M) * y.tiles_n;
    nY.push_back(y);
    GemmProb z{};
    z.M = x.s; z.N = x.w; z.K = x.L;
    z.a = x.XL; z.lda = x.L; z.b = x.Yt; z.ldb = x.L; z.c = x.Z2; z.ldc = x.w;
    z.kp = 1 | 2;       // XL and Yt blocked (K = L)
    z.a_bytes = (uint32_t)(2 * (size_t)x.s * x.L); z.b_bytes = (uint32_t)(2 * (size_t)x.w * x.L);
    z.tiles_n = gemm_nt_tiles_n(z.N); z.tile_start = tnz; tnz += gemm_nt_tiles_m(z.M) * z.tiles_n;
    if (use_qz) z.c_parts = x.Z2p;   // every Z2 but the last one feeds an early orthonormalisation
    nZ.push_back(z);
    // split iterations: V's bf16 parts v_m, v_l (both orientations), the iterates' residuals.
    // The operator V is kept to about 2^-24 (v_h + v_m + v_l), the iterates Z^T and Y^T to
    // 2^-17 (a perturbation of the iterate, which later iterations damp, not of the
    // operator): five products, h.h + l.h + h.m + l.m + h.l (iterate.operator); the
    // three-product form drops the last two (operator kept to 2^-17 only).
    SplitProb sp{};
    sp.g = (const float*)grads[x.idx]; sp.inv = c.decompose ? h.inv : nullptr; sp.inv_ld = h.k;
    sp.B = c.block_size; sp.m = h.m; sp.n = h.n;
    const bool rgt = h.side == MOARA_SIDE_RIGHT;   // m x n is X_K (RIGHT) or X_L (LEFT)
    sp.out_n[0] = rgt ? x.VKm : x.XLm; sp.out_n[1] = rgt ? x.VKl : x.XLl;
    sp.out_t[0] = rgt ? x.XLm : x.VKm; sp.out_t[1] = rgt ? x.XLl : x.VKl;
    sp.tiles_c = (int32_t)((h.n + 63) / 64); sp.tile_start = tvlo; tvlo += split_lo_tiles(h.m, h.n);
    vlo.push_back(sp);
    a.out_lo = x.Ztlo;   // same tiles as tZ
    tZs.push_back(a);
    auto segs = [](GemmProb& g, int terms, const void* it_h, const void* it_l, const void* op_h, const void* op_m,
                   const void* op_l, bool it_is_a) {
      const void* it[5] = {it_h, it_l, it_h, it_l, it_h};
      const void* op[5] = {op_h, op_h, op_m, op_m, op_l};
      g.nseg = terms;
      for (int j = 0; j < 5; ++j) {
        const void* pa = it_is_a ? it[j] : op[j];
        const void* pb = it_is_a ? op[j] : it[j];
        if (j == 0) { g.a = pa; g.b = pb; } else if (j < terms) { g.seg_a[j - 1] = pa; g.seg_b[j - 1] = pb; }
      }
    };
    GemmProb y3 = y;   // Y^T = Z^T X_K^T: iterate Zt (A), operator X_K (B); Yt split on output
    segs(y, 5, x.Zt, x.Ztlo, h.V, x.VKm, x.VKl, true);
    segs(y3, 3, x.Zt, x.Ztlo, h.V, x.VKm, x.VKl, true);
    y.c_lo = y3.c_lo = x.Ytlo;
    nYs.push_back(y);
    nYs3.push_back(y3);
    GemmProb z3 = z;   // Z2 = X_L Y: operator X_L (A), iterate Yt (B)
    segs(z, 5, x.Yt, x.Ytlo, x.XL, x.XLm, x.XLl, false);
    segs(z3, 3, x.Yt, x.Ytlo, x.XL, x.XLm, x.XLl, false);
    nZs.push_back(z);
    nZs3.push_back(z3);
    // last iteration: Y (L x w, fp32 for its CholeskyQR) = X_K Z, split
    GemmProb f{};
    f.M = x.L; f.N = x.w; f.K = x.s;
    f.lda = x.s; f.ldb = x.s;
    segs(f, 5, x.Zt, x.Ztlo, h.V, x.VKm, x.VKl, false);
    f.c = x.Y; f.ldc = x.w;
    f.kp = 1 | 2;
    f.a_bytes = (uint32_t)(2 * (size_t)x.L * x.s); f.b_bytes = (uint32_t)(2 * (size_t)x.w * x.s);
    f.tiles_n = gemm_nt_tiles_n(f.N); f.tile_start = tnyf; tnyf += gemm_nt_tiles_m(f.M) * f.tiles_n;
    nYf.push_back(f);
    // ... and its orthonormalised Y2 split into three bf16 parts of Y^T (w x L, blocked, K = L)
    // for the last product Z2 = X_L Y2, where a perturbation of the iterate is no longer
    // damped (it moves span(Z2) by about its size times sigma_1 / sigma_r): six products,
    // operator . iterate h.h + h.m + m.h + h.l + m.m + l.h (both kept to about 2^-24)
    GemmProb zf = z;
    zf.c_parts = nullptr;
    {
      const void* op[6] = {x.XL, x.XL, x.XLm, x.XL, x.XLm, x.XLl};
      const void* it[6] = {x.Yt, x.Ytlo, x.Yt, x.Ytl2, x.Ytlo, x.Yt};
      zf.a = op[0]; zf.b = it[0]; zf.nseg = 6;
      for (int j = 1; j < 6; ++j) { zf.seg_a[j - 1] = op[j]; zf.seg_b[j - 1] = it[j]; }
    }
    nZf.push_back(zf);
    TransProb q2{};
    q2.in = x.Y2; q2.out = x.Yt; q2.out_lo = x.Ytlo; q2.out_lo2 = x.Ytl2;
    q2.rows = x.L; q2.cols = x.w; q2.ldi = x.w; q2.ldo = x.L;
    q2.in_f32 = 1; q2.out_kp = 1;
    q2.tiles_c = (int32_t)((x.w + 63) / 64); q2.tile_start = tty2; tty2 += transpose_tiles(x.L, x.w);
    if (use_qz) {
      // (R^{-1})^T in three bf16 parts, blocked (rows w, K = w): A of the product below
      TransProb tr{};
      const size_t ww = (size_t)x.w * x.w;
      tr.in = x.Rinv; tr.out = x.Rtp; tr.out_lo = (bf16*)x.Rtp + ww; tr.out_lo2 = (bf16*)x.Rtp + 2 * ww;
      tr.rows = x.w; tr.cols = x.w; tr.ldi = x.w; tr.ldo = x.w; tr.in_f32 = 1; tr.out_kp = 1;
      tr.tiles_c = (int32_t)((x.w + 63) / 64); tr.tile_start = ttr; ttr += transpose_tiles(x.w, x.w);
      tR.push_back(tr);
      // Z^T = (R^{-1})^T Z2^T: A = (R^{-1})^T, lower triangular (A[n][k] = 0 for k > n, so a
      // tile's K loop ends at its last row), B = Z2 (rows s, K = w); six part products
      // h.h + h.m + m.h + h.l + l.h + m.m; output Z^T in bf16, blocked (K = s)
      GemmProb g{};
      g.M = x.w; g.N = x.s; g.K = x.w;
      g.lda = x.w; g.ldb = x.w; g.c = x.Zt; g.ldc = x.s;
      g.kp = 1 | 2 | 4;
      g.tri_b = 2;
      g.a_bytes = (uint32_t)(2 * ww); g.b_bytes = (uint32_t)(2 * (size_t)x.s * x.w);
      const bf16* ra = (const bf16*)x.Rtp;
      const bf16* zb = (const bf16*)x.Z2p;
      const size_t sw = (size_t)x.s * x.w;
      const void* pa[6] = {ra, ra, ra + ww, ra, ra + 2 * ww, ra + ww};
      const void* pb[6] = {zb, zb + sw, zb, zb + 2 * sw, zb, zb + sw};
      g.a = pa[0]; g.b = pb[0]; g.nseg = 6;
      for (int j = 1; j < 6; ++j) { g.seg_a[j - 1] = pa[j]; g.seg_b[j - 1] = pb[j]; }
      g.tiles_n = gemm_nt_tiles_n(g.N); g.tile_start = tqz; tqz += gemm_nt_tiles_m(g.M) * g.tiles_n;
      qZ.push_back(g);
      g.c_lo = x.Ztlo;   // before a split iteration: also the residual part of Z^T
      qZs.push_back(g);
    }
    tY2.push_back(q2);
  }

  struct Part { const void* p; size_t b; };
  std::vector<Part> parts = {
      {rd.data(), sizeof(RefDev) * nm},                               // 0
      {gZ2.first.data(), sizeof(GramProb) * nm},                      // 1
      {gY.first.data(), sizeof(GramProb) * nm},                       // 2
      {aZ.first.data(), sizeof(GemmProb) * nm},                       // 3
      {aY.first.data(), sizeof(GemmProb) * nm},                       // 4
      {xzR.first.data(), sizeof(GemmProb) * xzR.first.size()},       // 5
      {xzL.first.data(), sizeof(GemmProb) * xzL.first.size()},       // 6
      {xtR.first.data(), sizeof(GemmProb) * xtR.first.size()},       // 7
      {xtL.first.data(), sizeof(GemmProb) * xtL.first.size()},       // 8
      {xt2R.first.data(), sizeof(GemmProb) * xt2R.first.size()},     // 9
      {xt2L.first.data(), sizeof(GemmProb) * xt2L.first.size()},     // 10
      {pan_pref.data(), sizeof(uint32_t) * pan_pref.size()},          // 11
      {upd_pref.data(), sizeof(uint32_t) * upd_pref.size()},          // 12
      {inv_pref.data(), sizeof(uint32_t) * inv_pref.size()},          // 13
      {vlo.data(), sizeof(SplitProb) * vlo.size()},                   // 14
      {tZs.data(), sizeof(TransProb) * tZs.size()},                   // 15
      {nYs.data(), sizeof(GemmProb) * nYs.size()},                    // 16
      {nZs.data(), sizeof(GemmProb) * nZs.size()},                    // 17
      {tZ.data(), sizeof(TransProb) * tZ.size()},                     // 18
      {tX.data(), sizeof(TransProb) * tX.size()},                     // 19
      {nY.data(), sizeof(GemmProb) * nY.size()},                      // 20
      {nZ.data(), sizeof(GemmProb) * nZ.size()},                      // 21
      {pwl.data(), sizeof(GemmProb) * pwl.size()},                    // 22
      {nYf.data(), sizeof(GemmProb) * nYf.size()},                    // 23
      {tY2.data(), sizeof(TransProb) * tY2.size()},                   // 24
      {nYs3.data(), sizeof(GemmProb) * nYs3.size()},                  // 25
      {nZs3.data(), sizeof(GemmProb) * nZs3.size()},                  // 26
      {nZf.data(), sizeof(GemmProb) * nZf.size()},                    // 27
      {tR.data(), sizeof(TransProb) * tR.size()},                     // 28
      {qZ.data(), sizeof(GemmProb) * qZ.size()},                      // 29
      {qZs.data(), sizeof(GemmProb) * qZs.size()},                    // 30
      {aZf.first.data(), sizeof(GemmProb) * aZf.first.size()},       // 31
  };
  size_t total = 0;
  std::vector<size_t> offs;
  for (auto& pp : parts) { offs.push_back(total); total += align_up(pp.b ? pp.b : 1); }
  if (total > st->ref_arena_bytes && st->noalloc)
    return fail(MOARA_E_UNSUPPORTED, "refresh descriptors of %zu bytes exceed the no-alloc scratch (%zu bytes)", total,
                st->ref_arena_bytes);
  if (total > st->ref_arena_bytes) {
    HIP_TRY(hipStreamSynchronize(stream));
    if (st->ref_arena) (void)hipFree(st->ref_arena);
    if (st->ref_host) (void)hipHostFree(st->ref_host);
    st->ref_arena = nullptr; st->ref_host = nullptr; st->ref_arena_bytes = 0;
    if (hipMalloc(&st->ref_arena, total) != hipSuccess) return fail(MOARA_E_OOM, "refresh descriptor arena");
    if (hipHostMalloc(&st->ref_host, total) != hipSuccess) return fail(MOARA_E_OOM, "refresh pinned arena");
    st->ref_arena_bytes = total;
  }
  // the pinned buffer and arena are shared by all refresh chunks: wait for earlier users
  HIP_TRY(hipStreamSynchronize(stream));
  if (st->noalloc) {
    // no pinned buffer of our own: copy from ordinary host memory and wait for the copy
    std::vector<char> hb(total);
    for (size_t q = 0; q < parts.size(); ++q)
      if (parts[q].b) memcpy(hb.data() + offs[q], parts[q].p, parts[q].b);
    HIP_TRY(hipMemcpyAsync(st->ref_arena, hb.data(), total, hipMemcpyHostToDevice, stream));
    HIP_TRY(hipStreamSynchronize(stream));
  } else {
    for (size_t q = 0; q < parts.size(); ++q)
      if (parts[q].b) memcpy(st->ref_host + offs[q], parts[q].p, parts[q].b);
    HIP_TRY(hipMemcpyAsync(st->ref_arena, st->ref_host, total, hipMemcpyHostToDevice, stream));
  }
  auto D = [&](int q) { return (const void*)(st->ref_arena + offs[q]); };
  const RefDev* RD = (const RefDev*)D(0);

  auto gemm = [&](int am, int q, const std::pair<std::vector<GemmProb>, uint32_t>& l) -> hipError_t {
    if (l.first.empty()) return hipSuccess;
    return launch_gemm(kind, am, B_NC, EP_STORE, (const GemmProb*)D(q), (int)l.first.size(), l.second, u, stream);
  };
  const uint32_t* PAN = (const uint32_t*)D(11);
  const uint32_t* UPD = (const uint32_t*)D(12);
  const uint32_t* INV = (const uint32_t*)D(13);
  auto chol_inv = [&]() -> hipError_t {      // C -> R (in place), X = R^{-1}, Rinv = fp32(X)
    hipError_t e = hipSuccess;
    for (int k = 0; k < nbmax && e == hipSuccess; ++k) {
      e = k == 0 ? launch_chol_diag(RD, nm, stream) : launch_chol_row(RD, UPD + (size_t)k * nm, nm, upd_tot[k], k, stream);
      if (e == hipSuccess) e = launch_chol_panel(RD, PAN + (size_t)k * nm, nm, pan_tot[k], k, stream);
    }
    for (int l = 1; l <= nlev && e == hipSuccess; ++l)
      for (int ph = 0; ph < 2 && e == hipSuccess; ++ph)
        e = launch_trtri(RD, INV + (size_t)(l - 1) * nm, nm, inv_tot[l - 1], l, ph, stream);
    return e;
  };
  // Z <- orth(Z2). An early one (more iterations follow) forms the bf16-path matrices'
  // next Z^T (and its residual part before a split iteration) directly; the fp32 Z
  // is then formed for the other matrices only.
  bool zt_ready = false;
  auto orth_Z = [&](bool early, bool next_split) -> hipError_t {
    hipError_t e = launch_gram((const GramProb*)D(1), nm, gZ2.second, stream);
    if (e == hipSuccess) e = chol_inv();
    zt_ready = early && use_qz;
    if (!zt_ready) return e == hipSuccess ? gemm(A_KC, 3, aZ) : e;
    if (e == hipSuccess) e = gemm(A_KC, 31, aZf);
    if (e == hipSuccess) e = launch_transpose((const TransProb*)D(28), (int)tR.size(), ttr, stream);
    if (e == hipSuccess)
      e = launch_gemm_nt(EP_STORE_BF16, (const GemmProb*)D(next_split ? 30 : 29), (int)qZ.size(), tqz, u, stream);
    return e;
  };
  TimerScope ts(st, MOARA_KERN_REFRESH, stream);
  // the Gaussian start block; the same launch zeroes Rinv (its blocks below the diagonal
  // are never written by the factorisation kernels) and the per-sweep Jacobi measures
  HIP_TRY(launch_gauss(RD, nm, tg, stream));
  const int q_iters = c.refresh_iters;
  const int q_bf = q_iters > REFRESH_F32_ITERS ? q_iters - REFRESH_F32_ITERS : 0;
  if (orth0) HIP_TRY(orth_Z(false, false));   // the Gaussian block has no bf16 parts
  if (!nY.empty()) {
    HIP_TRY(launch_transpose((const TransProb*)D(19), (int)tX.size(), ttx, stream));
    HIP_TRY(launch_split_lo((const SplitProb*)D(14), (int)vlo.size(), tvlo, stream));
  }
  for (int it = 0; it < q_iters; ++it) {
    const bool last = it + 1 == q_iters;
    // fp32 products for the matrices without a bf16 V. Y = X Z : RIGHT X = V -> rows of G ;
    // LEFT X = V^T -> columns of G
    HIP_TRY(gemm(A_G_ROW, 5, xzR));
    HIP_TRY(gemm(A_G_TRANS, 6, xzL));
    if (!last) {
      HIP_TRY(gemm(A_G_TRANS, 7, xtR));
      HIP_TRY(gemm(A_G_ROW, 8, xtL));
    }
    // bf16 MFMA products for the others: plain in the early iterations, split (operands
    // and their residuals) in the last ones
    if (!nY.empty()) {
      if (it < q_bf) {
        if (!zt_ready) HIP_TRY(launch_transpose((const TransProb*)D(18), (int)tZ.size(), ttz, stream));
        HIP_TRY(launch_gemm_nt(EP_STORE_BF16, (const GemmProb*)D(20), (int)nY.size(), tny, u, stream));
        HIP_TRY(launch_gemm_nt(EP_STORE, (const GemmProb*)D(21), (int)nZ.size(), tnz, u, stream));
      } else {
        if (!zt_ready) HIP_TRY(launch_transpose((const TransProb*)D(15), (int)tZs.size(), ttz, stream));
        if (!last) {
          const bool five = it + REFRESH_SPLIT5_ITERS >= q_iters;
          HIP_TRY(launch_gemm_nt(EP_STORE_BF16, (const GemmProb*)D(five ? 16 : 25), (int)nYs.size(), tny, u, stream));
          HIP_TRY(launch_gemm_nt(EP_STORE, (const GemmProb*)D(five ? 17 : 26), (int)nZs.size(), tnz, u, stream));
        } else {
          HIP_TRY(launch_gemm_nt(EP_STORE, (const GemmProb*)D(23), (int)nYf.size(), tnyf, u, stream));
        }
      }
    }
    if (!last) {
      HIP_TRY(orth_Z(true, it + 1 >= q_bf));
    } else {   // Y2 = orth(Y) ; Z2 = X^T Y2
      HIP_TRY(launch_gram((const GramProb*)D(2), nm, gY.second, stream));
      HIP_TRY(chol_inv());
      HIP_TRY(gemm(A_KC, 4, aY));
      HIP_TRY(gemm(A_G_TRANS, 9, xt2R));
      HIP_TRY(gemm(A_G_ROW, 10, xt2L));
      if (!nY.empty()) {
        HIP_TRY(launch_transpose((const TransProb*)D(24), (int)tY2.size(), tty2, stream));
        HIP_TRY(launch_gemm_nt(EP_STORE, (const GemmProb*)D(27), (int)nZf.size(), tnz, u, stream));
      }
    }
  }
  // Rayleigh-Ritz: Z2 = Q R (CholeskyQR), SVD of the w x w factor R by one-sided Jacobi
  // (R J has orthogonal columns, norms = Ritz values), Ritz vectors Q (R J) / norm
  HIP_TRY(orth_Z(false, false));
  HIP_TRY(launch_r_colmajor(RD, nm, tc, stream));
  for (int sw = 0; sw < MAX_SWEEPS; ++sw)
    for (int rr = 0; rr < nb_max - 1; ++rr) HIP_TRY(launch_jacobi_round(RD, nm, tj, rr, sw, stream));
  HIP_TRY(launch_finalize_order(RD, nm, tnorm, stream));
  HIP_TRY(launch_gemm(kind, A_KC, B_KC, EP_STORE, (const GemmProb*)D(22), nm, tpw, u, stream));
  int32_t rmax = 0;
  for (auto& x : rm) rmax = std::max(rmax, st->mats[x.idx].r);
  HIP_TRY(launch_finalize_out(RD, nm, rmax, stream));
  HIP_TRY(launch_complete_basis(RD, nm, stream));
  for (auto& x : rm) st->mats[x.idx].hasP = st->mats[x.idx].refreshed = true;
  return MOARA_OK;
}

// Device bytes per refresh chunk. One chunk per refresh is fastest (the latency-bound
// Cholesky chains and Jacobi rounds then cover every matrix in one launch sequence):
// a Llama-2-7B-shaped stack needs about 131 GB (the split operands of the last
// iterations are 52 GB of it), under half of one MI355X's 288 GB. A refresh never plans
// a chunk larger than the device's free memory (plus the workspace it already holds),
// and callers cap it with MOARA_REFRESH_CHUNK_MIB (the projectors do not depend on the
// chunks).
#ifndef MOARA_REFRESH_BUDGET_GIB
#define MOARA_REFRESH_BUDGET_GIB 128
#endif
constexpr size_t REFRESH_BUDGET = (size_t)MOARA_REFRESH_BUDGET_GIB << 30;

// Chunk budget: REFRESH_BUDGET, or MOARA_REFRESH_CHUNK_MIB (MiB) from the environment
// when that is set to a positive integer (callers short of device memory; tests use it
// to run one refresh in several chunks).
size_t refresh_budget() {
  const char* e = getenv("MOARA_REFRESH_CHUNK_MIB");
  if (e && *e) {
    char* end = nullptr;
    const long long v = strtoll(e, &end, 10);
    if (end && *end == 0 && v > 0) return (size_t)v << 20;
  }
  return REFRESH_BUDGET;
}

// Upper bound of one refresh chunk's descriptor bytes (refresh_chunk's parts: RefDev,
// two Gram lists, the GEMM, transpose and split lists and the Cholesky and inverse
// prefix arrays, each part aligned).
size_t ref_desc_bound(size_t nm, int nbmax) {
  const int nlev = std::max(1, trtri_levels(nbmax));
  return 33 * ALIGN + nm * (sizeof(RefDev) + 2 * sizeof(GramProb) + 17 * sizeof(GemmProb) + 5 * sizeof(TransProb) +
                            sizeof(SplitProb) + 4 * (2 * (size_t)nbmax + (size_t)nlev));
}

// Refresh the matrices idx in order, in chunks whose workspace stays within the budget
// (a matrix larger than the budget forms a chunk of its own). Without allocation the
// budget is the scratch array's workspace part, and a chunk's descriptors must also fit
// its descriptor part.
int refresh_in_chunks(moara_state* st, const std::vector<int>& idx, const void* const* grads, hipStream_t stream,
                      const std::vector<char>& usev) {
  const bool na = st->noalloc;
  size_t budget = na ? st->ref_ws_bytes : refresh_budget();
  if (!na) {
    // never plan chunks larger than the device can hold now: the free memory plus the
    // workspace this state already owns (which a larger chunk would replace), less 1 GiB
    // for the caller (the projectors do not depend on how the matrices are chunked)
    size_t free_b = 0, total_b = 0;
    if (hipMemGetInfo(&free_b, &total_b) == hipSuccess) {
      const size_t usable = free_b + st->ref_ws_bytes;
      const size_t margin = (size_t)1 << 30;
      budget = std::min(budget, usable > margin ? usable - margin : (size_t)0);
    }
  }
  std::vector<int> chunk;
  size_t bytes = 0;
  int nbm = 1;
  int rc;
  for (int i : idx) {
    const MatHost& h = st->mats[i];
    const int32_t w = subspace_width(st->cfg, h.s, h.r);
    const size_t b = mat_refresh_bytes(h.s, h.L, w, h.r, usev[i]);
    const int nbm2 = std::max(nbm, chol_blocks(w));
    if (!chunk.empty() &&
        (bytes + b > budget || (na && ref_desc_bound(chunk.size() + 1, nbm2) > st->ref_arena_bytes))) {
      if ((rc = refresh_chunk(st, chunk, grads, stream, &usev))) return rc;
      chunk.clear();
      bytes = 0;
      nbm = 1;
    }
    chunk.push_back(i);
    bytes += b;
    nbm = std::max(nbm, chol_blocks(w));
  }
  return refresh_chunk(st, chunk, grads, stream, &usev);
}

// For the duration of one moara_step_noalloc call, the state's descriptor arena,
// refresh descriptor arena and refresh workspace are views into the scratch array:
//   [0, A)               step descriptors (A = the state's arena size)
//   [A, A + RD)          refresh descriptors of one chunk
//   [A + RD, capacity)   refresh workspace
// Timing events are off (creating them could allocate). Restored on exit.
struct NoallocView {
  moara_state* st;
  bool on;
  char *arena = nullptr, *ws = nullptr, *ra = nullptr;
  size_t wsb = 0, rab = 0;
  bool timing = false;
  NoallocView(moara_state* s, char* base, bool enable) : st(s), on(enable) {
    if (!on) return;
    arena = st->dev_arena; ws = st->ref_ws; wsb = st->ref_ws_bytes; ra = st->ref_arena; rab = st->ref_arena_bytes;
    timing = st->timing;
    const size_t A = align_up(st->arena_bytes);
    st->dev_arena = base;
    st->ref_arena = base + A;
    st->ref_arena_bytes = NOALLOC_REF_DESC_BYTES;
    st->ref_ws = base + A + NOALLOC_REF_DESC_BYTES;
    st->ref_ws_bytes = NOALLOC_SCRATCH_BYTES - A - NOALLOC_REF_DESC_BYTES;
    st->timing = false;
    st->noalloc = true;
  }
  ~NoallocView() {
    if (!on) return;
    st->dev_arena = arena; st->ref_ws = ws; st->ref_ws_bytes = wsb; st->ref_arena = ra; st->ref_arena_bytes = rab;
    st->timing = timing;
    st->noalloc = false;
  }
};

int run_refresh(moara_state* st, const std::vector<int>& idx, const void* const* grads, hipStream_t stream) {
  if (idx.empty()) return MOARA_OK;
  std::vector<char> usev(st->n, 0);
  for (int i : idx) usev[i] = st->mats[i].vpath && (((uintptr_t)grads[i] & 15) == 0);
  int rc = run_decompose(st, idx, grads, false, stream, &usev);
  if (rc) return rc;
  return refresh_in_chunks(st, idx, grads, stream, usev);
}

}  // namespace

// ============================================================================ ABI
extern "C" {

int moara_default_config(moara_config* out) {
  if (!out) return fail(MOARA_E_ARG, "out is NULL");
  memset(out, 0, sizeof *out);
  out->block_size = 128;
  out->beta1 = 0.9f;
  out->beta2 = 0.999f;
  out->adam_eps = 1e-6f;
  out->decomp_eps = 1e-12f;
  out->scale = 0.25f;
  out->weight_decay = 0.f;
  out->refresh_interval = 200;
  out->bias_correction = 1;
  out->decompose = 1;
  out->weight_dtype = MOARA_BF16;
  out->grad_dtype = MOARA_F32;
  out->operand_dtype = MOARA_BF16;
  out->refresh_oversample = -1;
  out->refresh_iters = 20;
  out->refresh_seed = 0;
  out->zero_grad_mode = 0;
  out->moment_dtype = MOARA_F32;
  return MOARA_OK;
}


int moara_allocate_ranks(int32_t r_base, uint32_t types_mask, uint32_t donor_mask, uint32_t receiver_mask,
                         int32_t delta_r, int32_t out_rank_table[MOARA_NUM_MODULES]) {
  if (!out_rank_table) return fail(MOARA_E_ARG, "out_rank_table is NULL");
  const uint32_t all = (1u << MOARA_NUM_MODULES) - 1u;
  if (types_mask == 0 || (types_mask & ~all)) return fail(MOARA_E_ARG, "types_mask must be a non-empty set of module ids");
  if ((donor_mask & ~types_mask) || (receiver_mask & ~types_mask))
    return fail(MOARA_E_ARG, "donor and receiver sets must be subsets of the module types");
  if (donor_mask & receiver_mask) return fail(MOARA_E_ARG, "donor and receiver sets overlap");
  if ((donor_mask == 0) != (receiver_mask == 0)) return fail(MOARA_E_ARG, "donor and receiver sets must both be empty or both non-empty");
  if (r_base < 1) return fail(MOARA_E_ARG, "r_base must be >= 1");
  if (delta_r < 0) return fail(MOARA_E_ARG, "delta_r must be >= 0");
  const int64_t nd = __builtin_popcount(donor_mask), nr = __builtin_popcount(receiver_mask);
  int64_t gain = 0;
  if (nr) {
    if (((int64_t)delta_r * nd) % nr != 0)
      return fail(MOARA_E_RANK, "receiver share delta_r*|D|/|R| = %d*%lld/%lld is not an integer", delta_r, (long long)nd, (long long)nr);
    gain = (int64_t)delta_r * nd / nr;
  }
  int32_t tmp[MOARA_NUM_MODULES];
  for (int t = 0; t < MOARA_NUM_MODULES; ++t) {
    int64_t r = 0;
    if (types_mask & (1u << t)) {
      if (donor_mask & (1u << t)) r = (int64_t)r_base - delta_r;
      else if (receiver_mask & (1u << t)) r = (int64_t)r_base + gain;
      else r = r_base;
      if (r < 1) return fail(MOARA_E_RANK, "rank of module %d falls below 1", t);
      if (r > INT32_MAX) return fail(MOARA_E_RANK, "rank of module %d overflows", t);
    }
    tmp[t] = (int32_t)r;
  }
  memcpy(out_rank_table, tmp, sizeof tmp);
  return MOARA_OK;
}

int moara_resolve_matrix(const moara_config* cfg, const moara_matrix_desc* desc, int32_t* out_rank, int32_t* out_side) {
  return resolve(cfg, desc, out_rank, out_side);
}

static int validate_all(const moara_config* cfg, const moara_matrix_desc* descs, int32_t n,
                        std::vector<int32_t>* ranks, std::vector<int32_t>* sides) {
  int rc = validate_config(cfg);
  if (rc) return rc;
  if (n < 1) return fail(MOARA_E_ARG, "n must be >= 1");
  if (!descs) return fail(MOARA_E_ARG, "descs is NULL");
  ranks->resize(n);
  sides->resize(n);
  for (int i = 0; i < n; ++i) {
    rc = resolve(cfg, &descs[i], &(*ranks)[i], &(*sides)[i]);
    if (rc) {
      g_err = "matrix " + std::to_string(i) + ": " + g_err;
      return rc;
    }
  }
  return MOARA_OK;
}

int moara_state_bytes(const moara_config* cfg, const moara_matrix_desc* descs, int32_t n, int64_t* out_state_bytes,
                      int64_t* out_refresh_workspace_bytes) {
  std::vector<int32_t> ranks, sides;
  int rc = validate_all(cfg, descs, n, &ranks, &sides);
  if (rc) return rc;
  if (!out_state_bytes) return fail(MOARA_E_ARG, "out_state_bytes is NULL");
  size_t tot = 0, ref = 0;
  for (int i = 0; i < n; ++i) {
    const Layout l = layout_of(descs[i], sides[i], cfg->block_size);
    tot += mat_state_bytes(*cfg, descs[i].rows, descs[i].cols, sides[i], l.s, l.L, l.k, ranks[i]);
    ref += mat_refresh_bytes(l.s, l.L, subspace_width(*cfg, l.s, ranks[i]), ranks[i],
                             vpath_shape_ok(*cfg, descs[i].rows, descs[i].cols, sides[i], ranks[i]));
  }
  tot += align_up(16 * (size_t)n);   // refresh records
  *out_state_bytes = (int64_t)tot;
  if (out_refresh_workspace_bytes) *out_refresh_workspace_bytes = (int64_t)std::min(ref, refresh_budget() + ref / (size_t)n);
  return MOARA_OK;
}

static void free_state(moara_state* st) {
  if (!st) return;
  // teardown: a failure to release one resource does not stop the release of the others
  if (st->block) (void)hipFree(st->block);
  if (st->dev_arena) (void)hipFree(st->dev_arena);
  if (st->host_ring) (void)hipHostFree(st->host_ring);
  if (st->ref_ws) (void)hipFree(st->ref_ws);
  if (st->ref_arena) (void)hipFree(st->ref_arena);
  if (st->ref_host) (void)hipHostFree(st->ref_host);
  for (auto& e : st->slot_ev)
    if (e) (void)hipEventDestroy(e);
  if (st->order_ev) (void)hipEventDestroy(st->order_ev);
  for (auto& tl : st->pending) { (void)hipEventDestroy(tl.a); (void)hipEventDestroy(tl.b); }
  for (auto e : st->ev_pool) (void)hipEventDestroy(e);
  delete st;
}

int moara_create_state(const moara_config* cfg, const moara_matrix_desc* descs, int32_t n, void* stream,
                       moara_state** out) {
  if (!out) return fail(MOARA_E_ARG, "out is NULL");
  *out = nullptr;
  std::vector<int32_t> ranks, sides;
  int rc = validate_all(cfg, descs, n, &ranks, &sides);
  if (rc) return rc;
  hipStream_t hs = (hipStream_t)stream;
  moara_state* st = new moara_state();
  st->cfg = *cfg;
  st->n = n;
  if (hipGetDevice(&st->device) != hipSuccess) { free_state(st); return fail(MOARA_E_HIP, "hipGetDevice failed (no GPU?)"); }
  if ((rc = scratch_init(st->device))) { free_state(st); return rc; }   // this GPU's scratch address, once
  st->mats.resize(n);
  size_t tot = 0;
  for (int i = 0; i < n; ++i) {
    const Layout l = layout_of(descs[i], sides[i], cfg->block_size);
    MatHost& h = st->mats[i];
    h.m = descs[i].rows; h.n = descs[i].cols; h.r = ranks[i]; h.side = sides[i];
    h.s = l.s; h.L = l.L; h.k = (int32_t)l.k;
    h.vpath = vpath_shape_ok(*cfg, h.m, h.n, h.side, h.r);
    h.kp = h.vpath && cfg->operand_dtype == MOARA_BF16 && h.r % 32 == 0;
    tot += mat_state_bytes(*cfg, h.m, h.n, h.side, h.s, h.L, h.k, h.r);
  }
  tot += align_up(16 * (size_t)n);   // refresh records
  if (hipMalloc(&st->block, tot) != hipSuccess) { free_state(st); return fail(MOARA_E_OOM, "state of %zu bytes", tot); }
  st->block_bytes = tot;
  const int ob = elem_bytes(cfg->operand_dtype);
  char* p = st->block;
  auto take = [&](size_t b) { char* q = p; p += align_up(b); return q; };
  for (auto& h : st->mats) {
    h.inv = (float*)take(4 * h.m * h.k);
    h.dM = (float*)take(4 * h.m * h.k);
    h.mag1 = (float*)take(4 * h.m * h.k);
    h.mag2 = (float*)take(4 * h.m * h.k);
    h.exp1 = take((size_t)elem_bytes(cfg->moment_dtype) * h.L * h.r);
    h.exp2 = take((size_t)elem_bytes(cfg->moment_dtype) * h.L * h.r);
    h.N = take((size_t)ob * h.L * h.r);
    h.P32 = (float*)take(4 * h.s * h.r);
    h.Pop = take((size_t)ob * h.s * h.r);
    h.Ptop = take((size_t)ob * h.s * h.r);
    if (h.vpath) h.V = take(2 * (size_t)h.m * h.n);
  }
  st->info_dev = (int32_t*)take(16 * (size_t)n);
  st->arena_bytes = 2 * align_up(sizeof(MatDev) * n) + 5 * align_up(sizeof(GemmProb) * n) + 8 * ALIGN;
  if (hipMalloc(&st->dev_arena, st->arena_bytes) != hipSuccess ||
      hipHostMalloc(&st->host_ring, st->arena_bytes * moara_state::NSLOT) != hipSuccess) {
    free_state(st);
    return fail(MOARA_E_OOM, "descriptor arenas");
  }
  for (auto& e : st->slot_ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) { free_state(st); return fail(MOARA_E_HIP, "event create"); }
  if (hipEventCreateWithFlags(&st->order_ev, hipEventDisableTiming) != hipSuccess) { free_state(st); return fail(MOARA_E_HIP, "event create"); }
  if (hipMemsetAsync(st->block, 0, tot, hs) != hipSuccess || hipStreamSynchronize(hs) != hipSuccess) {
    free_state(st);
    return fail(MOARA_E_HIP, "zero fill of the state failed");
  }
  *out = st;
  return MOARA_OK;
}

static int collect_active(moara_state* st, const void* const* ptrs, const uint8_t* active, std::vector<int>* idx,
                          const char* what) {
  idx->clear();
  for (int i = 0; i < st->n; ++i) {
    if (active && !active[i]) continue;
    if (!ptrs[i]) return fail(MOARA_E_ARG, "%s[%d] is NULL for an active matrix", what, i);
    idx->push_back(i);
  }
  return MOARA_OK;
}

int moara_refresh_projector(moara_state* st, const void* const* grads, const uint8_t* active, void* stream) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (!grads) return fail(MOARA_E_ARG, "grads is NULL");
  std::vector<int> idx;
  int rc = collect_active(st, grads, active, &idx, "grads");
  if (rc) return rc;
  if (idx.empty()) return MOARA_OK;
  ORDER_ON(st, (hipStream_t)stream);
  return run_refresh(st, idx, grads, (hipStream_t)stream);
}

// Subspace alignment diagnostic (Section 3.2): decompose G (inv only), R^(T) = V' P with
// the fp32 master projector (projection GEMMs with a plain store), then the
// reconstruction GEMM P R (LEFT) / R Q^T (RIGHT) whose epilogue scales by Rep_B(M) and
// reduces <G, G_recon>, ||G_recon||^2 and ||G||^2 per matrix. fp32 operands throughout.
int moara_alignment(moara_state* st, const void* const* grads, const uint8_t* active, double* out_S, void* stream) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (!grads || !out_S) return fail(MOARA_E_ARG, "grads/out_S is NULL");
  std::vector<int> idx;
  int rc = collect_active(st, grads, active, &idx, "grads");
  if (rc) return rc;
  for (int i : idx)
    if (!st->mats[i].hasP) return fail(MOARA_E_STATE, "matrix %d has no projector (set one or refresh first)", i);
  if (idx.empty()) return MOARA_OK;
  hipStream_t hs = (hipStream_t)stream;
  ORDER_ON(st, hs);
  const bool dec = st->cfg.decompose != 0;
  if (dec && (rc = run_decompose(st, idx, grads, false, hs))) return rc;
  size_t need = 0;
  for (int i : idx) need += align_up(4 * (size_t)st->mats[i].L * st->mats[i].r);   // R^(T), L x r fp32
  const size_t red_off = need;
  need += align_up(8 * 3 * idx.size());
  if ((rc = ensure_ref_ws(st, need))) return rc;
  double* red = (double*)(st->ref_ws + red_off);
  std::vector<GemmProb> projR, projL, rec;
  uint32_t tR = 0, tL = 0, tr = 0;
  char* p = st->ref_ws;
  for (size_t q = 0; q < idx.size(); ++q) {
    const int i = idx[q];
    const MatHost& h = st->mats[i];
    const bool left = h.side == MOARA_SIDE_LEFT;
    float* R = (float*)p;
    p += align_up(4 * (size_t)h.L * h.r);
    GemmProb g{};   // R^(T) (L x r) = V' P, V' = V (RIGHT) or V^T (LEFT) formed from G and inv
    g.M = h.L; g.N = h.r; g.K = h.s;
    g.a = grads[i]; g.lda = h.n;
    g.inv = dec ? h.inv : nullptr; g.inv_ld = h.k;
    g.b = h.P32; g.ldb = h.r;
    g.c = R; g.ldc = h.r;
    g.tiles_n = gemm_tiles_n(KIND_F32, g.N);
    g.vec = vec_flags_g((const float*)grads[i], h.n) | (vec_flags_op(h.P32, h.r, 0) << 1);
    set_extents(g, 4 * (size_t)h.m * h.n, 4 * (size_t)h.n, 4 * (size_t)h.s * h.r, 4 * (size_t)h.r,
                g.inv ? 4 * (size_t)h.m * h.k : 0, 4 * (size_t)h.k);
    const uint32_t nt = gemm_tiles_m(KIND_F32, g.M) * g.tiles_n;
    if (left) { g.tile_start = tL; tL += nt; projL.push_back(g); }
    else { g.tile_start = tR; tR += nt; projR.push_back(g); }
    GemmProb b{};   // reconstructed direction (m x n) = P R (LEFT) or R Q^T (RIGHT), reduced against G
    b.M = h.m; b.N = h.n; b.K = h.r;
    b.a = left ? (const void*)h.P32 : (const void*)R; b.lda = h.r;
    b.b = left ? (const void*)R : (const void*)h.P32; b.ldb = h.r;
    b.c = (void*)grads[i]; b.ldc = h.n;
    b.inv = dec ? h.inv : nullptr; b.inv_ld = h.k;
    b.red = red + 3 * q;
    b.tiles_n = gemm_tiles_n(KIND_F32, b.N);
    b.vec = vec_flags_op(b.a, h.r, 0) | (vec_flags_op(b.b, h.r, 0) << 1);
    set_extents(b, 4 * (size_t)h.m * h.r, 4 * (size_t)h.r, 4 * (size_t)h.n * h.r, 4 * (size_t)h.r, 0, 0);
    b.tile_start = tr;
    tr += gemm_tiles_m(KIND_F32, b.M) * b.tiles_n;
    rec.push_back(b);
  }
  Stager sg;
  if ((rc = begin_stage(st, sg))) return rc;
  const size_t oR = projR.empty() ? 0 : sg.push(projR.data(), projR.size());
  const size_t oL = projL.empty() ? 0 : sg.push(projL.data(), projL.size());
  const size_t oB = sg.push(rec.data(), rec.size());
  if (oR == (size_t)-1 || oL == (size_t)-1 || oB == (size_t)-1) return fail(MOARA_E_OOM, "descriptor arena too small");
  if ((rc = end_stage(st, sg, hs))) return rc;
  GemmUniform u = make_uniform(st, 0.f);
  u.decomp_eps = st->cfg.decomp_eps;
  {
    TimerScope ts(st, MOARA_KERN_ALIGN, hs);
    if (!projR.empty())
      HIP_TRY(launch_gemm(KIND_F32, A_G_ROW, B_NC, EP_STORE, (const GemmProb*)(st->dev_arena + oR), (int)projR.size(), tR, u, hs));
    if (!projL.empty())
      HIP_TRY(launch_gemm(KIND_F32, A_G_TRANS, B_NC, EP_STORE, (const GemmProb*)(st->dev_arena + oL), (int)projL.size(), tL, u, hs));
    HIP_TRY(hipMemsetAsync(red, 0, 8 * 3 * idx.size(), hs));
    HIP_TRY(launch_gemm(KIND_F32, A_KC, B_KC, EP_ALIGN, (const GemmProb*)(st->dev_arena + oB), (int)rec.size(), tr, u, hs));
  }
  std::vector<double> sums(3 * idx.size());
  HIP_TRY(hipMemcpyAsync(sums.data(), red, 8 * sums.size(), hipMemcpyDeviceToHost, hs));
  HIP_TRY(hipStreamSynchronize(hs));
  for (size_t q = 0; q < idx.size(); ++q) {
    const double den = sqrt(sums[3 * q + 1]) * sqrt(sums[3 * q + 2]);
    out_S[idx[q]] = den > 0.0 ? sums[3 * q] / den : 0.0;
  }
  return MOARA_OK;
}

static int step_impl(moara_state* st, void* const* weights, const void* const* grads, const uint8_t* active,
                     float lr, void* stream, bool noalloc) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (!weights || !grads) return fail(MOARA_E_ARG, "weights/grads is NULL");
  if (!isfinite(lr)) return fail(MOARA_E_ARG, "lr must be finite");
  std::vector<int> idx;
  int rc = collect_active(st, grads, active, &idx, "grads");
  if (rc) return rc;
  for (int i : idx)
    if (!weights[i]) return fail(MOARA_E_ARG, "weights[%d] is NULL for an active matrix", i);
  const int T = st->cfg.refresh_interval;
  std::vector<int> need;
  for (int i : idx) {
    const MatHost& h = st->mats[i];
    if (T > 0 && h.t % T == 0) need.push_back(i);
    else if (!h.hasP) return fail(MOARA_E_STATE, "matrix %d has no projector (set one, refresh, or use refresh_interval > 0)", i);
  }
  // zero_grad_mode 1: the inactive matrices take a step with G = 0 (their grads entries are not read)
  std::vector<int> zidx;
  std::vector<char> zflag(st->n, 0);
  if (st->cfg.zero_grad_mode == 1 && active) {
    for (int i = 0; i < st->n; ++i) {
      if (active[i]) continue;
      const MatHost& h = st->mats[i];
      if (!weights[i]) return fail(MOARA_E_ARG, "weights[%d] is NULL (zero_grad_mode 1 steps inactive matrices too)", i);
      if (!(T > 0 && h.t % T == 0) && !h.hasP)
        return fail(MOARA_E_STATE, "matrix %d has no projector (set one, refresh, or use refresh_interval > 0)", i);
      zidx.push_back(i);
      zflag[i] = 1;
    }
  }
  if (idx.empty() && zidx.empty()) return MOARA_OK;
  hipStream_t hs = (hipStream_t)stream;
  char* base = nullptr;
  if (noalloc) {
    // every limit is checked before anything is enqueued
    base = (st->device >= 0 && st->device < MAX_DEVICES) ? g_scratch_ptr[st->device] : nullptr;
    if (!base) return fail(MOARA_E_STATE, "no scratch address for device %d", st->device);
    const size_t A = align_up(st->arena_bytes);
    if (A + NOALLOC_REF_DESC_BYTES >= NOALLOC_SCRATCH_BYTES)
      return fail(MOARA_E_UNSUPPORTED, "the state's step descriptors (%zu bytes) do not fit the no-alloc scratch", A);
    const size_t wcap = NOALLOC_SCRATCH_BYTES - A - NOALLOC_REF_DESC_BYTES;
    for (int i : need) {
      const MatHost& h = st->mats[i];
      const int32_t w = subspace_width(st->cfg, h.s, h.r);
      const bool bf = h.vpath && (((uintptr_t)grads[i] & 15) == 0);
      const size_t b = mat_refresh_bytes(h.s, h.L, w, h.r, bf);
      if (b > wcap)
        return fail(MOARA_E_UNSUPPORTED,
                    "matrix %d (%lld x %lld, r = %d) needs a refresh workspace of %zu bytes, more than the %zu bytes "
                    "the no-alloc scratch holds (refresh it with moara_step or moara_refresh_projector)",
                    i, (long long)h.m, (long long)h.n, h.r, b, wcap);
    }
  }
  ORDER_ON(st, hs);
  if (noalloc && g_scratch_ev_valid[st->device]) HIP_TRY(hipStreamWaitEvent(hs, g_scratch_ev[st->device], 0));
  NoallocView view(st, base, noalloc);
  std::vector<char> usev(st->n, 0);
  for (int i : idx) usev[i] = st->mats[i].vpath && (((uintptr_t)grads[i] & 15) == 0);
  if (st->cfg.decompose) {
    rc = run_decompose(st, idx, grads, true, hs, &usev);
    if (rc) return rc;
  }
  if (!need.empty() && (rc = refresh_in_chunks(st, need, grads, hs, usev))) return rc;
  if ((rc = run_zero_grad(st, zidx, hs))) return rc;
  std::vector<int> all = idx;
  all.insert(all.end(), zidx.begin(), zidx.end());
  rc = run_project_back(st, all, weights, grads, lr, hs, &usev, &zflag);
  if (rc) return rc;
  for (int i : all) st->mats[i].t += 1;
  if (noalloc) {
    HIP_TRY(hipEventRecord(g_scratch_ev[st->device], hs));
    g_scratch_ev_valid[st->device] = true;
  }
  return MOARA_OK;
}

int moara_step(moara_state* st, void* const* weights, const void* const* grads, const uint8_t* active, float lr,
               void* stream) {
  return step_impl(st, weights, grads, active, lr, stream, false);
}

int moara_step_noalloc(moara_state* st, void* const* weights, const void* const* grads, const uint8_t* active,
                       float lr, void* stream) {
  return step_impl(st, weights, grads, active, lr, stream, true);
}

static int tensor_geometry(moara_state* st, int32_t mat, int32_t which, size_t* bytes) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (mat < 0 || mat >= st->n) return fail(MOARA_E_ARG, "matrix index %d out of range", mat);
  const MatHost& h = st->mats[mat];
  switch (which) {
    case MOARA_T_P: *bytes = 4 * h.s * h.r; break;
    case MOARA_T_EXP_AVG:
    case MOARA_T_EXP_AVG_SQ: *bytes = 4 * h.L * h.r; break;
    case MOARA_T_MAG_AVG:
    case MOARA_T_MAG_AVG_SQ: *bytes = 4 * h.m * h.k; break;
    case MOARA_T_STEP: *bytes = 8; break;
    default: return fail(MOARA_E_ARG, "unknown tensor id %d", which);
  }
  return MOARA_OK;
}

int moara_get_tensor(moara_state* st, int32_t mat, int32_t which, void* host_dst, size_t bytes, void* stream) {
  size_t need = 0;
  int rc = tensor_geometry(st, mat, which, &need);
  if (rc) return rc;
  if (!host_dst) return fail(MOARA_E_ARG, "host_dst is NULL");
  if (bytes != need) return fail(MOARA_E_SHAPE, "buffer is %zu bytes, tensor needs %zu", bytes, need);
  const MatHost& h = st->mats[mat];
  if (which == MOARA_T_STEP) { memcpy(host_dst, &h.t, 8); return MOARA_OK; }
  if (which == MOARA_T_P && !h.hasP) return fail(MOARA_E_STATE, "matrix %d has no projector yet", mat);
  hipStream_t hs = (hipStream_t)stream;
  const void* src = which == MOARA_T_P ? (const void*)h.P32
                  : which == MOARA_T_EXP_AVG ? (const void*)h.exp1
                  : which == MOARA_T_EXP_AVG_SQ ? (const void*)h.exp2
                  : which == MOARA_T_MAG_AVG ? (const void*)h.mag1 : (const void*)h.mag2;
  const bool moment = which == MOARA_T_EXP_AVG || which == MOARA_T_EXP_AVG_SQ;
  const bool transpose = moment && h.side == MOARA_SIDE_LEFT;
  const bool narrow = moment && st->cfg.moment_dtype == MOARA_BF16;
  ORDER_ON(st, hs);
  HIP_TRY(hipStreamSynchronize(hs));
  if (!transpose && !narrow) {
    HIP_TRY(hipMemcpyAsync(host_dst, src, need, hipMemcpyDeviceToHost, hs));
    HIP_TRY(hipStreamSynchronize(hs));
    return MOARA_OK;
  }
  const size_t cnt = (size_t)h.L * h.r;
  std::vector<float> tmp(cnt);
  if (narrow) {
    std::vector<uint16_t> raw(cnt);
    HIP_TRY(hipMemcpyAsync(raw.data(), src, 2 * cnt, hipMemcpyDeviceToHost, hs));
    HIP_TRY(hipStreamSynchronize(hs));
    for (size_t i = 0; i < cnt; ++i) tmp[i] = host_bf16_to_f32(raw[i]);
  } else {
    HIP_TRY(hipMemcpyAsync(tmp.data(), src, need, hipMemcpyDeviceToHost, hs));
    HIP_TRY(hipStreamSynchronize(hs));
  }
  float* o = (float*)host_dst;
  if (!transpose) {
    memcpy(o, tmp.data(), need);
    return MOARA_OK;
  }
  // paper orientation r x n from the stored n x r
  for (int64_t l = 0; l < h.L; ++l)
    for (int64_t j = 0; j < h.r; ++j) o[j * h.L + l] = tmp[l * h.r + j];
  return MOARA_OK;
}

int moara_set_tensor(moara_state* st, int32_t mat, int32_t which, const void* host_src, size_t bytes, void* stream) {
  size_t need = 0;
  int rc = tensor_geometry(st, mat, which, &need);
  if (rc) return rc;
  if (!host_src) return fail(MOARA_E_ARG, "host_src is NULL");
  if (bytes != need) return fail(MOARA_E_SHAPE, "buffer is %zu bytes, tensor needs %zu", bytes, need);
  MatHost& h = st->mats[mat];
  if (which == MOARA_T_STEP) {
    int64_t t;
    memcpy(&t, host_src, 8);
    if (t < 0) return fail(MOARA_E_ARG, "step counter must be >= 0");
    h.t = t;
    return MOARA_OK;
  }
  hipStream_t hs = (hipStream_t)stream;
  void* dst = which == MOARA_T_P ? (void*)h.P32
            : which == MOARA_T_EXP_AVG ? (void*)h.exp1
            : which == MOARA_T_EXP_AVG_SQ ? (void*)h.exp2
            : which == MOARA_T_MAG_AVG ? (void*)h.mag1 : (void*)h.mag2;
  const bool moment = which == MOARA_T_EXP_AVG || which == MOARA_T_EXP_AVG_SQ;
  const bool transpose = moment && h.side == MOARA_SIDE_LEFT;
  const bool narrow = moment && st->cfg.moment_dtype == MOARA_BF16;
  std::vector<float> tmp;
  std::vector<uint16_t> raw;
  const void* src = host_src;
  size_t dev_bytes = need;
  if (transpose) {
    tmp.resize((size_t)h.L * h.r);
    const float* in = (const float*)host_src;
    for (int64_t l = 0; l < h.L; ++l)
      for (int64_t j = 0; j < h.r; ++j) tmp[l * h.r + j] = in[j * h.L + l];
    src = tmp.data();
  }
  if (narrow) {
    const size_t cnt = (size_t)h.L * h.r;
    const float* in = (const float*)src;
    raw.resize(cnt);
    for (size_t i = 0; i < cnt; ++i) raw[i] = host_f32_to_bf16(in[i]);
    src = raw.data();
    dev_bytes = 2 * cnt;
  }
  ORDER_ON(st, hs);
  HIP_TRY(hipStreamSynchronize(hs));
  HIP_TRY(hipMemcpyAsync(dst, src, dev_bytes, hipMemcpyHostToDevice, hs));
  if (which == MOARA_T_P) {
    HIP_TRY(launch_convert_projector(h.P32, h.Pop, h.Ptop, h.s, h.r, st->cfg.operand_dtype == MOARA_BF16, h.kp ? 1 : 0,
                                     hs));
    h.hasP = true;
  }
  HIP_TRY(hipStreamSynchronize(hs));
  return MOARA_OK;
}

int moara_refresh_info(moara_state* st, int32_t mat, int32_t* out_sweeps, int32_t* out_converged,
                       int32_t* out_rank, float* out_offdiag, void* stream) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (mat < 0 || mat >= st->n) return fail(MOARA_E_ARG, "matrix index %d out of range", mat);
  if (!st->mats[mat].refreshed) return fail(MOARA_E_STATE, "matrix %d has not been refreshed by the library", mat);
  hipStream_t hs = (hipStream_t)stream;
  int32_t rec[4];
  ORDER_ON(st, hs);
  HIP_TRY(hipStreamSynchronize(hs));
  HIP_TRY(hipMemcpy(rec, st->info_dev + 4 * (size_t)mat, sizeof rec, hipMemcpyDeviceToHost));
  if (out_sweeps) *out_sweeps = rec[0];
  if (out_converged) *out_converged = rec[1];
  if (out_rank) *out_rank = rec[2];
  if (out_offdiag) memcpy(out_offdiag, &rec[3], 4);
  return MOARA_OK;
}

int moara_set_timing(moara_state* st, int32_t enable) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  st->timing = enable != 0;
  return MOARA_OK;
}

int moara_kernel_stats(moara_state* st, int32_t kernel, int64_t* out_launches, double* out_total_ms, void* stream) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (kernel < 0 || kernel >= MOARA_NUM_KERNELS) return fail(MOARA_E_ARG, "kernel id %d out of range", kernel);
  int rc = collect_timing(st, (hipStream_t)stream);
  if (rc) return rc;
  if (out_launches) *out_launches = st->launches[kernel];
  if (out_total_ms) *out_total_ms = st->total_ms[kernel];
  return MOARA_OK;
}

int moara_reset_kernel_stats(moara_state* st, void* stream) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  int rc = collect_timing(st, (hipStream_t)stream);
  if (rc) return rc;
  for (int k = 0; k < MOARA_NUM_KERNELS; ++k) { st->launches[k] = 0; st->total_ms[k] = 0.0; }
  return MOARA_OK;
}

int moara_matrix_info(const moara_state* st, int32_t mat, int64_t* rows, int64_t* cols, int32_t* rank, int32_t* side,
                      int32_t* n_blocks) {
  if (!st) return fail(MOARA_E_ARG, "state is NULL");
  if (mat < 0 || mat >= st->n) return fail(MOARA_E_ARG, "matrix index %d out of range", mat);
  const MatHost& h = st->mats[mat];
  if (rows) *rows = h.m;
  if (cols) *cols = h.n;
  if (rank) *rank = h.r;
  if (side) *side = h.side;
  if (n_blocks) *n_blocks = h.k;
  return MOARA_OK;
}

void moara_destroy_state(moara_state* st) {
  if (!st) return;
  // every call that enqueued work on the state recorded order_ev last: waiting for it
  // waits for all of the state's work, on whichever streams it ran
  if (st->order_valid) (void)hipEventSynchronize(st->order_ev);
  free_state(st);
}

const char* moara_last_error(void) { return g_err.c_str(); }

const char* moara_version(void) { return "moara-mi355x 0.1 (gfx950)"; }

}  // extern "C"
