// api.hip -- the C ABI of libilw.so (declared in include/ilw.h): argument
// validation on the host before anything is launched, workspace layout, and
// kernel launches on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "ilw_internal.h"

using namespace ilw;

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

int ok() {
  g_err.clear();
  return ILW_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(ILW_E_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

// ---- per-stage timing (tracing) ------------------------------------------
struct ProfRecord {
  int stage;
  hipEvent_t start, stop;
};
// The tracing state is shared by every thread: the switch is an atomic read
// on every launch, the event pool and the records are guarded by the mutex.
struct Profiler {
  std::mutex mu;
  std::atomic<bool> on{false};
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<ProfRecord> recs;
} g_prof;

hipEvent_t prof_event() {  // with g_prof.mu held
  if (g_prof.used == g_prof.pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_prof.pool.push_back(e);
  }
  return g_prof.pool[g_prof.used++];
}

// Brackets one kernel launch with events when profiling is enabled.
struct StageTimer {
  int stage;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  StageTimer(int st, hipStream_t str) : stage(st), s(str) {
    if (!g_prof.on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    a = prof_event();
    b = prof_event();
    if (a && b) (void)hipEventRecord(a, s);
  }
  void done() {
    if (!a || !b) return;
    std::lock_guard<std::mutex> lk(g_prof.mu);
    (void)hipEventRecord(b, s);
    g_prof.recs.push_back({stage, a, b});
  }
};

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ---- static scratch of ilw_block_forward_noalloc -------------------------
// One file-scope device array; every GPU that loads the library holds its
// own copy at its own address.  Host code never passes the array's name to a
// kernel (on the host it is only a stand-in for the symbol): it uses the
// device address looked up once per device, with that device current.
static __device__ __align__(256) int8_t scratch[ILW_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int8_t* g_scratch_addr[kMaxDevices];

int scratch_of_current_device(int8_t** out) {
  int dev = -1;
  hipError_t he = hipGetDevice(&dev);
  if (he != hipSuccess) return fail(ILW_E_HIP, "hipGetDevice: %s", hipGetErrorString(he));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(ILW_E_UNSUPPORTED, "device ordinal %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* addr = nullptr;
    he = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (he != hipSuccess || !addr)
      return fail(ILW_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                  hipGetErrorString(he));
    g_scratch_addr[dev] = (int8_t*)addr;
  }
  *out = g_scratch_addr[dev];
  return ILW_OK;
}

#define REQUIRE(cond, code, ...)            \
  do {                                      \
    if (!(cond)) return fail(code, __VA_ARGS__); \
  } while (0)

int check_dyadic(const ilw_dyadic& d, int32_t channels, const char* name) {
  REQUIRE(d.mult && d.shift, ILW_E_NULL, "%s: mult/shift must not be NULL", name);
  REQUIRE(d.n == 1 || d.n == channels, ILW_E_SHAPE,
          "%s: n = %d must be 1 (per-tensor) or %d (per-channel)", name, d.n, channels);
  return ILW_OK;
}

int check_shift(int32_t s, const char* name) {
  REQUIRE(s >= 1 && s <= 62, ILW_E_PARAM, "%s = %d must be in [1, 62]", name, s);
  return ILW_OK;
}

int check_mult(int32_t m, const char* name) {
  REQUIRE(m != INT32_MIN, ILW_E_PARAM, "%s must not be INT32_MIN", name);
  return ILW_OK;
}

int check_shiftmax(int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p, int32_t s_d) {
  REQUIRE(I0 >= 1 && I0 < (1 << 14), ILW_E_PARAM, "I0 = %d must be in [1, 2^14 - 1]", I0);
  REQUIRE(k_inter >= 1 && k_inter <= 16, ILW_E_PARAM, "k_inter = %d must be in [1, 16]",
          k_inter);
  REQUIRE(k_out >= 2 && k_out <= 8, ILW_E_PARAM, "k_out = %d must be in [2, 8]", k_out);
  REQUIRE(m_p >= 0 && m_p <= 31, ILW_E_PARAM, "m_p = %d must be in [0, 31]", m_p);
  REQUIRE(s_d >= -1 && s_d <= 31, ILW_E_PARAM, "s_d = %d must be -1 or in [0, 31]", s_d);
  return ILW_OK;
}

int check_gelu(int32_t I0, int32_t k_inter, int32_t k_out, int32_t mult, int32_t shift) {
  REQUIRE(I0 >= 1 && I0 < (1 << 14), ILW_E_PARAM, "GELU I0 = %d must be in [1, 2^14 - 1]",
          I0);
  REQUIRE(k_inter >= 1 && k_inter <= 16, ILW_E_PARAM, "GELU k_inter = %d must be in [1, 16]",
          k_inter);
  REQUIRE(k_out >= 2 && k_out <= 8, ILW_E_PARAM, "GELU k_out = %d must be in [2, 8]", k_out);
  int e;
  if ((e = check_mult(mult, "GELU out_mult"))) return e;
  return check_shift(shift, "GELU out_shift");
}

// Geometry of window or global attention over a grid.
struct Geometry {
  int32_t T, nwx, nW, wh, ww, Tw, Twp;
};

int check_geometry(int32_t batch, int32_t gh, int32_t gw, int32_t wh, int32_t ww,
                   Geometry* g) {
  REQUIRE(batch >= 0, ILW_E_SHAPE, "batch = %d must be >= 0", batch);
  REQUIRE(gh >= 1 && gw >= 1, ILW_E_SHAPE, "grid %dx%d must be positive", gh, gw);
  REQUIRE((int64_t)gh * gw <= (1 << 24), ILW_E_SHAPE, "grid %dx%d too large", gh, gw);
  if (wh == 0 && ww == 0) {
    wh = gh;
    ww = gw;
  }
  REQUIRE(wh >= 1 && ww >= 1 && gh % wh == 0 && gw % ww == 0, ILW_E_SHAPE,
          "window %dx%d must tile the %dx%d grid", wh, ww, gh, gw);
  g->T = gh * gw;
  g->wh = wh;
  g->ww = ww;
  g->nwx = gw / ww;
  g->nW = (gh / wh) * g->nwx;
  g->Tw = wh * ww;
  REQUIRE(g->Tw <= 2048, ILW_E_UNSUPPORTED, "%d tokens per window exceed the 2048 limit",
          g->Tw);
  REQUIRE((int64_t)batch * g->T < ((int64_t)1 << 23), ILW_E_UNSUPPORTED,
          "batch * tokens = %lld must be below 2^23", (long long)batch * g->T);
  REQUIRE((int64_t)batch * g->nW <= 65535, ILW_E_UNSUPPORTED,
          "batch * windows = %lld exceeds 65535", (long long)batch * g->nW);
  g->Twp = (g->Tw + 63) & ~63;
  return ILW_OK;
}

int check_attn(const ilw_attn_params* ap) {
  REQUIRE(ap, ILW_E_NULL, "attention parameters must not be NULL");
  int e;
  if ((e = check_mult(ap->score_mult, "score_mult"))) return e;
  if ((e = check_shift(ap->score_shift, "score_shift"))) return e;
  if ((e = check_mult(ap->pv_mult, "pv_mult"))) return e;
  if ((e = check_shift(ap->pv_shift, "pv_shift"))) return e;
  return check_shiftmax(ap->I0, ap->k_inter, ap->k_out, ap->m_p, ap->s_d);
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// base + off inside a workspace; a null base (a size query) stays null, since
// an offset from a null pointer is undefined.
int8_t* carve(int8_t* base, size_t off) { return base ? base + off : nullptr; }

// Window-major Q/K/V^T buffers carved from a workspace.
size_t qkv_bytes(int32_t batch, const Geometry& g, int32_t D, QkvLayout* L, int8_t* base,
                 int32_t hd = 64) {
  const int32_t H = D / hd;
  const size_t qk = (size_t)batch * g.nW * H * g.Tw * 64;
  const size_t vt = (size_t)batch * g.nW * H * 64 * g.Twp;
  if (L) {
    L->q = base;
    L->k = carve(base, align256(qk));
    L->vt = carve(base, 2 * align256(qk));
    L->T = g.T;
    L->D = D;
    L->H = H;
    L->grid_w = g.nwx * g.ww;
    L->win_h = g.wh;
    L->win_w = g.ww;
    L->nwx = g.nwx;
    L->nW = g.nW;
    L->Tw = g.Tw;
    L->Twp = g.Twp;
    L->hs = hd == 32 ? 5 : 6;
  }
  return 2 * align256(qk) + align256(vt);
}

AttnArgs attn_args(const QkvLayout& L, int8_t* out, int32_t batch,
                   const ilw_attn_params& ap) {
  AttnArgs a;
  a.q = L.q;
  a.k = L.k;
  a.vt = L.vt;
  a.out = out;
  a.B = batch;
  a.T = L.T;
  a.D = L.D;
  a.H = L.H;
  a.grid_w = L.grid_w;
  a.win_h = L.win_h;
  a.win_w = L.win_w;
  a.nwx = L.nwx;
  a.nW = L.nW;
  a.Tw = L.Tw;
  a.Twp = L.Twp;
  a.score_mult = ap.score_mult;
  a.score_shift = ap.score_shift;
  a.I0 = ap.I0;
  a.k_inter = ap.k_inter;
  a.k_out = ap.k_out;
  a.m_p = ap.m_p;
  a.s_d = ap.s_d;
  a.pv_mult = ap.pv_mult;
  a.pv_shift = ap.pv_shift;
  a.hd = 1 << L.hs;
  return a;
}

GemmArgs gemm_args(const int8_t* x, const int8_t* w, const int32_t* b, const ilw_dyadic& d,
                   int8_t* y, int64_t M, int32_t N, int32_t K) {
  GemmArgs a = {};
  a.x = x;
  a.w = w;
  a.bias = b;
  a.mult = d.mult;
  a.shift = d.shift;
  a.nq = d.n;
  a.M = M;
  a.N = N;
  a.K = K;
  a.y = y;
  return a;
}

struct BlockLayout {
  QkvLayout qkv;
  int8_t *h, *att, *x1, *g;
  // proj and fc2 weights packed in MFMA fragment order for the 384-channel
  // LayerNorm-fused kernel, or null where that kernel does not run
  int8_t *wp_proj, *wp_fc2, *wp_fc1;
  size_t total;
};

bool ln_fusable(int32_t D);

// Where everything after attention runs as one packed-weight kernel (dim
// 384; ILW_FUSE_TAIL=0 turns it off, read once) the projection, fc1 and fc2
// weights are packed.
bool packs_fc1(const ilw_block_params* p, int64_t M) {
  static const bool on = [] {  // thread-safe static initialisation
    const char* e = getenv("ILW_FUSE_TAIL");
    return !(e && e[0] == '0');
  }();
  return on && ln_fusable(p->dim) && tail384_kernel_applies(M, p->dim, p->mlp_dim);
}
// Otherwise the 384-channel residual linears past the GEMM latency mode take
// the packed-weight LayerNorm kernel: the projection (its LayerNorm is LN2)
// and fc2 (with the next block's LN1, or without a LayerNorm after the last
// block).
bool packs_proj(const ilw_block_params* p, int64_t M) {
  return packs_fc1(p, M) ||
         (ln_fusable(p->dim) && ln384_packed_kernel_applies(M, p->dim, p->dim));
}
bool packs_fc2(const ilw_block_params* p, int64_t M) {
  return packs_fc1(p, M) ||
         (ln_fusable(p->dim) && ln384_packed_kernel_applies(M, p->dim, p->mlp_dim));
}
size_t packed_bytes(const ilw_block_params* p, int64_t M) {
  return (packs_proj(p, M) ? align256(packed_frag_bytes(p->dim, p->dim)) : 0) +
         (packs_fc2(p, M) ? align256(packed_frag_bytes(p->dim, p->mlp_dim)) : 0) +
         (packs_fc1(p, M) ? align256(packed_frag_bytes(p->mlp_dim, p->dim)) : 0);
}
// Carves the packed weights of a block from base + off; returns the bytes used.
size_t packed_layout(const ilw_block_params* p, int64_t M, int8_t* base, size_t off,
                     BlockLayout* L) {
  size_t used = 0;
  L->wp_proj = L->wp_fc2 = L->wp_fc1 = nullptr;
  if (packs_proj(p, M)) {
    L->wp_proj = carve(base, off);
    used += align256(packed_frag_bytes(p->dim, p->dim));
  }
  if (packs_fc2(p, M)) {
    L->wp_fc2 = carve(base, off + used);
    used += align256(packed_frag_bytes(p->dim, p->mlp_dim));
  }
  if (packs_fc1(p, M)) {
    L->wp_fc1 = carve(base, off + used);
    used += align256(packed_frag_bytes(p->mlp_dim, p->dim));
  }
  return used;
}
// One launch packing the listed blocks' weights (in groups of kMaxPack).
hipError_t pack_block_weights(const ilw_block_params* const* ps, const BlockLayout* Ls, int32_t n,
                              hipStream_t s) {
  PackList pl = {};
  auto flush = [&]() -> hipError_t {
    if (pl.n == 0) return hipSuccess;
    const hipError_t e = launch_pack_frags(pl, s);
    pl = PackList{};
    return e;
  };
  auto add = [&](const int8_t* src, int8_t* dst, int32_t N, int32_t K) -> hipError_t {
    if (pl.n == kMaxPack) {
      const hipError_t e = flush();
      if (e != hipSuccess) return e;
    }
    pl.src[pl.n] = src;
    pl.dst[pl.n] = dst;
    pl.K[pl.n] = K;
    pl.start[pl.n + 1] = pl.start[pl.n] + (int64_t)N * K / 16;
    ++pl.n;
    return hipSuccess;
  };
  for (int32_t b = 0; b < n; ++b) {
    hipError_t e = hipSuccess;
    if (Ls[b].wp_proj) e = add(ps[b]->w_proj, Ls[b].wp_proj, ps[b]->dim, ps[b]->dim);
    if (e == hipSuccess && Ls[b].wp_fc2)
      e = add(ps[b]->w_fc2, Ls[b].wp_fc2, ps[b]->dim, ps[b]->mlp_dim);
    if (e == hipSuccess && Ls[b].wp_fc1)
      e = add(ps[b]->w_fc1, Ls[b].wp_fc1, ps[b]->mlp_dim, ps[b]->dim);
    if (e != hipSuccess) return e;
  }
  return flush();
}

// Workspace of one block: h | Q K V^T | att | x1 | g.  qkv_reserve (when
// larger than this block's need) fixes the size of the Q K V^T region, so
// that in an encoder every block's att buffer lies past every block's Q K V^T.
size_t block_layout(const ilw_block_params* p, int32_t batch, const Geometry& g,
                    int8_t* base, BlockLayout* out, size_t qkv_reserve = 0,
                    bool with_packed = true) {
  const size_t M = (size_t)batch * g.T;
  size_t off = 0;
  BlockLayout L;
  L.h = carve(base, off);
  off += align256(M * p->dim);
  size_t q = qkv_bytes(batch, g, p->dim, &L.qkv, carve(base, off));
  off += q > qkv_reserve ? q : qkv_reserve;
  L.att = carve(base, off);
  off += align256(M * p->dim);
  L.x1 = carve(base, off);
  off += align256(M * p->dim);
  L.g = carve(base, off);
  off += align256(M * p->mlp_dim);
  // a single block has no next block: its fc2 takes the plain residual tile
  L.wp_proj = L.wp_fc2 = L.wp_fc1 = nullptr;
  if (with_packed) off += packed_layout(p, (int64_t)M, base, off, &L);
  L.total = off;
  if (out) *out = L;
  return off;
}

int check_block(const ilw_block_params* p, int32_t batch, int32_t gh, int32_t gw,
                int32_t wh, int32_t ww, Geometry* g) {
  REQUIRE(p, ILW_E_NULL, "block parameters must not be NULL");
  REQUIRE(p->head_dim == 64, ILW_E_UNSUPPORTED, "head_dim = %d: only 64 is implemented",
          p->head_dim);
  REQUIRE(p->heads >= 1 && p->dim == p->heads * p->head_dim, ILW_E_SHAPE,
          "dim = %d must equal heads (%d) * head_dim", p->dim, p->heads);
  REQUIRE(p->dim % 16 == 0 && p->mlp_dim >= 16 && p->mlp_dim % 16 == 0, ILW_E_SHAPE,
          "dim = %d and mlp_dim = %d must be multiples of 16", p->dim, p->mlp_dim);
  REQUIRE(p->mlp_dim <= 65536 && p->dim <= 16384, ILW_E_UNSUPPORTED,
          "dim/mlp_dim too large");
  REQUIRE(p->ln_iters >= 1 && p->ln_iters <= 64, ILW_E_PARAM,
          "ln_iters = %d must be in [1, 64]", p->ln_iters);
  REQUIRE(p->ln1_beta && p->ln2_beta, ILW_E_NULL, "LayerNorm beta must not be NULL");
  REQUIRE(p->w_qkv && p->w_proj && p->w_fc1 && p->w_fc2, ILW_E_NULL,
          "weights must not be NULL");
  REQUIRE(aligned16(p->w_qkv) && aligned16(p->w_proj) && aligned16(p->w_fc1) &&
              aligned16(p->w_fc2),
          ILW_E_PARAM, "weights must be 16-byte aligned");
  int e;
  if ((e = check_dyadic(p->ln1_out, p->dim, "ln1_out"))) return e;
  if ((e = check_dyadic(p->ln2_out, p->dim, "ln2_out"))) return e;
  if ((e = check_dyadic(p->qkv, 3 * p->dim, "qkv"))) return e;
  if ((e = check_dyadic(p->proj, p->dim, "proj"))) return e;
  if ((e = check_dyadic(p->fc1, p->mlp_dim, "fc1"))) return e;
  if ((e = check_dyadic(p->fc2, p->dim, "fc2"))) return e;
  if ((e = check_attn(&p->attn))) return e;
  if ((e = check_gelu(p->gelu_I0, p->gelu_k_inter, p->gelu_k_out, p->gelu_mult,
                      p->gelu_shift)))
    return e;
  if ((e = check_mult(p->res1_mult_a, "res1_mult_a")) || (e = check_mult(p->res1_mult_b, "res1_mult_b")) ||
      (e = check_shift(p->res1_shift, "res1_shift")) ||
      (e = check_mult(p->res2_mult_a, "res2_mult_a")) || (e = check_mult(p->res2_mult_b, "res2_mult_b")) ||
      (e = check_shift(p->res2_shift, "res2_shift")))
    return e;
  return check_geometry(batch, gh, gw, wh, ww, g);
}

// LayerNorm can be fused into the epilogue of the residual GEMM that
// produces its input when one workgroup holds whole rows: 3 or 6 waves of 64
// channels.
// ILW_FUSE_LN=0 runs every LayerNorm as its own kernel (same results; for
// comparisons), read once.
bool ln_fusable(int32_t D) {
  static const bool on = [] {  // read once (thread-safe static initialisation)
    const char* e = getenv("ILW_FUSE_LN");
    return !(e && e[0] == '0');
  }();
  return on && (D == 192 || D == 256 || D == 384);
}

GemmArgs with_ln(GemmArgs a, const int32_t* beta, const ilw_dyadic& out, int32_t iters,
                 int8_t* y2) {
  a.y2 = y2;
  a.ln_beta = beta;
  a.ln_mult = out.mult;
  a.ln_shift = out.shift;
  a.ln_nq = out.n;
  a.ln_iters = iters;
  return a;
}

// The block tail kernel (projection ... next block's QKV in one launch) covers
// dim 192 / MLP 768.  It pays off where launches dominate: by default for up
// to 8192 tokens per call; ILW_TAIL=0 / 1 turns it off / on wherever it
// applies (same results), read once.
bool use_tail(const ilw_block_params* p, const ilw_block_params* next, int64_t M) {
  static const int mode = [] {  // read once (thread-safe static initialisation)
    const char* e = getenv("ILW_TAIL");
    return (e && e[0] == '0') ? 0 : ((e && e[0] == '1') ? 1 : 2);
  }();
  if (mode == 0 || p->dim != 192 || p->mlp_dim != 768) return false;
  if (next && next->dim != 192) return false;
  // measured on the 1600-token encoder: the block tail wins up to batch 5,
  // the separate linears from batch 6
  return mode == 1 || M <= 8192;
}

// What the previous block already left for this one in the workspace.
enum { READY_NONE = 0, READY_H = 1, READY_QKV = 2 };

// One encoder block: h = LN1(x) and Q, K, V^T (unless already there),
// attention, then either the block tail kernel (which also leaves the next
// block's Q, K, V^T in next_qkv) or projection + residual (+ LN2), fc1 +
// GELU and fc2 + residual (+ the next block's LN1 in h).
int run_block(const ilw_block_params* p, const ilw_block_params* next,
              const QkvLayout* next_qkv, const int8_t* x, int8_t* y, int32_t batch,
              const Geometry& g, const BlockLayout& L, int ready, int* ready_out,
              hipStream_t s) {
  const int64_t M = (int64_t)batch * g.T;
  const int32_t D = p->dim, Hm = p->mlp_dim;
  const bool fuse = ln_fusable(D);
  hipError_t he = hipSuccess;
  *ready_out = READY_NONE;

  // h = LN1(x) and Q, K, V^T in one launch where the tail kernel runs
  if (ready == READY_NONE && use_tail(p, nullptr, M)) {
    TailArgs ha = {};
    ha.x = x;
    ha.M = M;
    ha.ln1_beta = p->ln1_beta; ha.ln1_mult = p->ln1_out.mult;
    ha.ln1_shift = p->ln1_out.shift; ha.ln1_nq = p->ln1_out.n; ha.ln1_iters = p->ln_iters;
    ha.w_qkv = p->w_qkv; ha.b_qkv = p->b_qkv; ha.qkv_mult = p->qkv.mult;
    ha.qkv_shift = p->qkv.shift; ha.qkv_nq = p->qkv.n;
    ha.qkv = L.qkv;
    StageTimer t(ILW_STAGE_GEMM_QKV, s);
    he = launch_block_head(ha, s);
    t.done();
    if (he != hipSuccess) return hip_status(he, "block LN1 + QKV");
    ready = READY_QKV;
  }
  // h = LN1(x)
  if (ready == READY_NONE) {
    StageTimer t(ILW_STAGE_LAYERNORM, s);
    he = launch_layernorm(x, L.h, M, D, p->ln1_beta, p->ln1_out.mult, p->ln1_out.shift,
                          p->ln1_out.n, p->ln_iters, s);
    t.done();
    if (he != hipSuccess) return hip_status(he, "block LN1");
  }
  // q, k, v^T = QKV(h), scattered window-major
  GemmArgs a;
  if (ready != READY_QKV) {
    a = gemm_args(L.h, p->w_qkv, p->b_qkv, p->qkv, nullptr, M, 3 * D, D);
    a.qkv = L.qkv;
    StageTimer t(ILW_STAGE_GEMM_QKV, s);
    he = launch_gemm(EPI_QKV, a, s);
    t.done();
    if (he != hipSuccess) return hip_status(he, "block QKV");
  }
  // att = Attn(q, k, v)
  {
    StageTimer t(ILW_STAGE_ATTENTION, s);
    he = launch_attention(attn_args(L.qkv, L.att, batch, p->attn), s);
    t.done();
  }
  if (he != hipSuccess) return hip_status(he, "block attention");

  if (use_tail(p, next_qkv ? next : nullptr, M)) {
    TailArgs ta = {};
    ta.att = L.att;
    ta.x = x;
    ta.y = y;
    ta.M = M;
    ta.w_proj = p->w_proj; ta.b_proj = p->b_proj; ta.proj_mult = p->proj.mult;
    ta.proj_shift = p->proj.shift; ta.proj_nq = p->proj.n;
    ta.res1_ma = p->res1_mult_a; ta.res1_mb = p->res1_mult_b; ta.res1_shift = p->res1_shift;
    ta.ln2_beta = p->ln2_beta; ta.ln2_mult = p->ln2_out.mult; ta.ln2_shift = p->ln2_out.shift;
    ta.ln2_nq = p->ln2_out.n; ta.ln2_iters = p->ln_iters;
    ta.w_fc1 = p->w_fc1; ta.b_fc1 = p->b_fc1; ta.fc1_mult = p->fc1.mult;
    ta.fc1_shift = p->fc1.shift; ta.fc1_nq = p->fc1.n;
    ta.g_I0 = p->gelu_I0; ta.g_kinter = p->gelu_k_inter; ta.g_kout = p->gelu_k_out;
    ta.g_mult = p->gelu_mult; ta.g_shift = p->gelu_shift;
    ta.w_fc2 = p->w_fc2; ta.b_fc2 = p->b_fc2; ta.fc2_mult = p->fc2.mult;
    ta.fc2_shift = p->fc2.shift; ta.fc2_nq = p->fc2.n;
    ta.res2_ma = p->res2_mult_a; ta.res2_mb = p->res2_mult_b; ta.res2_shift = p->res2_shift;
    if (next && next_qkv) {
      ta.has_next = 1;
      ta.ln1_beta = next->ln1_beta; ta.ln1_mult = next->ln1_out.mult;
      ta.ln1_shift = next->ln1_out.shift; ta.ln1_nq = next->ln1_out.n;
      ta.ln1_iters = next->ln_iters;
      ta.w_qkv = next->w_qkv; ta.b_qkv = next->b_qkv; ta.qkv_mult = next->qkv.mult;
      ta.qkv_shift = next->qkv.shift; ta.qkv_nq = next->qkv.n;
      ta.qkv = *next_qkv;
    }
    {
      StageTimer t(ILW_STAGE_BLOCK_TAIL, s);
      he = launch_block_tail(ta, s);
      t.done();
    }
    if (he != hipSuccess) return hip_status(he, "block tail");
    *ready_out = ta.has_next ? READY_QKV : READY_NONE;
    return ok();
  }

  if (L.wp_fc1) {
    // everything after attention in one launch: x1, h and g stay on chip
    GemmArgs fp = gemm_args(L.att, p->w_proj, p->b_proj, p->proj, L.x1, M, D, D);
    fp.wp = L.wp_proj;
    fp.resid = x;
    fp.res_ma = p->res1_mult_a;
    fp.res_mb = p->res1_mult_b;
    fp.res_shift = p->res1_shift;
    fp = with_ln(fp, p->ln2_beta, p->ln2_out, p->ln_iters, L.h);
    GemmArgs f1 = gemm_args(nullptr, p->w_fc1, p->b_fc1, p->fc1, L.g, M, Hm, D);
    f1.wp = L.wp_fc1;
    f1.g_I0 = p->gelu_I0;
    f1.g_kinter = p->gelu_k_inter;
    f1.g_kout = p->gelu_k_out;
    f1.g_mult = p->gelu_mult;
    f1.g_shift = p->gelu_shift;
    GemmArgs f2 = gemm_args(nullptr, p->w_fc2, p->b_fc2, p->fc2, y, M, D, Hm);
    f2.wp = L.wp_fc2;
    f2.res_ma = p->res2_mult_a;
    f2.res_mb = p->res2_mult_b;
    f2.res_shift = p->res2_shift;
    const bool ln = next && fuse;
    if (ln) f2 = with_ln(f2, next->ln1_beta, next->ln1_out, next->ln_iters, L.h);
    {
      StageTimer t(ILW_STAGE_TAIL384, s);
      he = launch_tail384(fp, f1, f2, ln, s);
      t.done();
    }
    if (he != hipSuccess) return hip_status(he, "block tail (dim 384)");
    *ready_out = ln ? READY_H : READY_NONE;
    return ok();
  }
  // x1 = Res(proj(att), x);  h = LN2(x1)
  a = gemm_args(L.att, p->w_proj, p->b_proj, p->proj, L.x1, M, D, D);
  a.wp = fuse ? L.wp_proj : nullptr;
  a.resid = x;
  a.res_ma = p->res1_mult_a;
  a.res_mb = p->res1_mult_b;
  a.res_shift = p->res1_shift;
  {
    StageTimer t(ILW_STAGE_GEMM_PROJ, s);
    he = fuse ? launch_gemm(EPI_RESID_LN, with_ln(a, p->ln2_beta, p->ln2_out, p->ln_iters, L.h), s)
              : launch_gemm(EPI_RESID, a, s);
    t.done();
  }
  if (he != hipSuccess) return hip_status(he, "block proj");
  if (!fuse) {
    StageTimer t(ILW_STAGE_LAYERNORM, s);
    he = launch_layernorm(L.x1, L.h, M, D, p->ln2_beta, p->ln2_out.mult, p->ln2_out.shift,
                          p->ln2_out.n, p->ln_iters, s);
    t.done();
    if (he != hipSuccess) return hip_status(he, "block LN2");
  }
  // g = rq(SD-ShiftGELU(fc1(h)))
  a = gemm_args(L.h, p->w_fc1, p->b_fc1, p->fc1, L.g, M, Hm, D);
  a.g_I0 = p->gelu_I0;
  a.g_kinter = p->gelu_k_inter;
  a.g_kout = p->gelu_k_out;
  a.g_mult = p->gelu_mult;
  a.g_shift = p->gelu_shift;
  {
    StageTimer t(ILW_STAGE_GEMM_FC1, s);
    he = launch_gemm(EPI_GELU, a, s);
    t.done();
  }
  if (he != hipSuccess) return hip_status(he, "block fc1");
  // y = Res(fc2(g), x1);  h = LN1'(y) of the next block
  a = gemm_args(L.g, p->w_fc2, p->b_fc2, p->fc2, y, M, D, Hm);
  a.wp = L.wp_fc2;  // set only where packs_fc2 holds
  a.resid = L.x1;
  a.res_ma = p->res2_mult_a;
  a.res_mb = p->res2_mult_b;
  a.res_shift = p->res2_shift;
  {
    StageTimer t(ILW_STAGE_GEMM_FC2, s);
    he = next && fuse
             ? launch_gemm(EPI_RESID_LN,
                           with_ln(a, next->ln1_beta, next->ln1_out, next->ln_iters, L.h), s)
             : launch_gemm(EPI_RESID, a, s);
    t.done();
  }
  if (he != hipSuccess) return hip_status(he, "block fc2");
  *ready_out = next && fuse ? READY_H : READY_NONE;
  return ok();
}

int check_encoder(const ilw_block_params* blocks, int32_t n_blocks, const int32_t* windows,
                  int32_t batch, int32_t grid_h, int32_t grid_w) {
  REQUIRE(blocks && windows, ILW_E_NULL, "blocks and windows (host) must not be NULL");
  REQUIRE(n_blocks >= 1 && n_blocks <= 4096, ILW_E_SHAPE, "n_blocks = %d must be in [1, 4096]",
          n_blocks);
  for (int32_t b = 0; b < n_blocks; ++b) {
    Geometry g;
    int e;
    if ((e = check_block(&blocks[b], batch, grid_h, grid_w, windows[2 * b],
                         windows[2 * b + 1], &g)))
      return e;
    REQUIRE(blocks[b].dim == blocks[0].dim, ILW_E_SHAPE,
            "block %d has dim %d, block 0 has %d: the residual stream width must not change",
            b, blocks[b].dim, blocks[0].dim);
  }
  return ILW_OK;
}

// Largest Q K V^T region over the blocks of an encoder.
size_t encoder_qkv_reserve(const ilw_block_params* blocks, int32_t n_blocks,
                           const int32_t* windows, int32_t batch, int32_t grid_h,
                           int32_t grid_w) {
  size_t q = 0;
  for (int32_t b = 0; b < n_blocks; ++b) {
    Geometry g;
    check_geometry(batch, grid_h, grid_w, windows[2 * b], windows[2 * b + 1], &g);
    const size_t n = qkv_bytes(batch, g, blocks[b].dim, nullptr, nullptr);
    q = n > q ? n : q;
  }
  return q;
}

size_t encoder_workspace(const ilw_block_params* blocks, int32_t n_blocks,
                         const int32_t* windows, int32_t batch, int32_t grid_h, int32_t grid_w) {
  const size_t q = encoder_qkv_reserve(blocks, n_blocks, windows, batch, grid_h, grid_w);
  size_t need = 0, packed = 0;
  for (int32_t b = 0; b < n_blocks; ++b) {
    Geometry g;
    check_geometry(batch, grid_h, grid_w, windows[2 * b], windows[2 * b + 1], &g);
    const size_t n = block_layout(&blocks[b], batch, g, nullptr, nullptr, q, false);
    need = n > need ? n : need;
    packed += packed_bytes(&blocks[b], (int64_t)batch * g.T);
  }
  // every block's packed weights after the shared per-block region
  return need + packed;
}

// The encoder's packed weights: block b's after those of blocks 0 .. b - 1,
// past the shared per-block region.
size_t encoder_shared_bytes(const ilw_block_params* blocks, int32_t n_blocks,
                            const int32_t* windows, int32_t batch, int32_t grid_h, int32_t grid_w) {
  const size_t q = encoder_qkv_reserve(blocks, n_blocks, windows, batch, grid_h, grid_w);
  size_t need = 0;
  for (int32_t b = 0; b < n_blocks; ++b) {
    Geometry g;
    check_geometry(batch, grid_h, grid_w, windows[2 * b], windows[2 * b + 1], &g);
    const size_t n = block_layout(&blocks[b], batch, g, nullptr, nullptr, q, false);
    need = n > need ? n : need;
  }
  return need;
}

// ---- decoder layer -------------------------------------------------------
struct DecoderLayout {
  QkvLayout qkv;
  int8_t *att, *x, *t1, *t2, *v, *off8, *lg, *smp, *g;
  size_t total;
};

size_t decoder_layout(const ilw_decoder_params* p, int32_t batch, int32_t Q, int32_t S,
                      int8_t* base, DecoderLayout* out) {
  Geometry g;
  check_geometry(batch, 1, Q, 0, 0, &g);
  const int32_t D = p->dim, NO = p->heads * p->levels * p->points * 2;
  const size_t MQ = (size_t)batch * Q, MS = (size_t)batch * S;
  DecoderLayout L;
  size_t off = 0;
  off += qkv_bytes(batch, g, D, &L.qkv, base, D / p->heads);
  auto take = [&](size_t bytes) {
    int8_t* ptr = carve(base, off);
    off += align256(bytes);
    return ptr;
  };
  L.att = take(MQ * D);
  L.x = take(MQ * D);
  L.t1 = take(MQ * D);
  L.t2 = take(MQ * D);
  L.v = take(MS * D);
  L.off8 = take(MQ * NO);
  L.lg = take(MQ * NO / 2);
  L.smp = take(MQ * D);
  L.g = take(MQ * p->ffn_dim);
  L.total = off;
  if (out) *out = L;
  return off;
}

int check_decoder(const ilw_decoder_params* p, int32_t batch, int32_t Q, int32_t S) {
  REQUIRE(p, ILW_E_NULL, "decoder parameters must not be NULL");
  REQUIRE(p->ref_dims == 2 || p->ref_dims == 4, ILW_E_PARAM,
          "ref_dims = %d: references are points (2) or boxes (4)", p->ref_dims);
  REQUIRE(p->heads >= 1 && p->dim >= 16 && p->dim % p->heads == 0, ILW_E_SHAPE,
          "dim = %d must be a multiple of heads = %d", p->dim, p->heads);
  const int32_t hd = p->dim / p->heads;
  REQUIRE(hd == 32 || hd == 64, ILW_E_UNSUPPORTED, "head_dim = %d: 32 and 64 are implemented",
          hd);
  REQUIRE(p->dim % 16 == 0 && p->ffn_dim >= 16 && p->ffn_dim % 16 == 0 &&
              p->dim <= 16384 && p->ffn_dim <= 65536,
          ILW_E_SHAPE, "dim = %d and ffn_dim = %d must be multiples of 16", p->dim,
          p->ffn_dim);
  REQUIRE(p->levels >= 1 && p->levels <= kMaxLevels && p->points >= 1 &&
              p->levels * p->points <= 64,
          ILW_E_SHAPE, "levels = %d, points = %d invalid", p->levels, p->points);
  REQUIRE((p->heads * p->levels * p->points) % 16 == 0, ILW_E_SHAPE,
          "heads*levels*points = %d must be a multiple of 16",
          p->heads * p->levels * p->points);
  REQUIRE(p->ln_iters >= 1 && p->ln_iters <= 64, ILW_E_PARAM,
          "ln_iters = %d must be in [1, 64]", p->ln_iters);
  REQUIRE(batch >= 0 && Q >= 1 && Q <= 2048 && S >= 1, ILW_E_SHAPE,
          "batch = %d, queries = %d (in [1, 2048]), value_tokens = %d invalid", batch, Q, S);
  REQUIRE((int64_t)batch * S < ((int64_t)1 << 31), ILW_E_UNSUPPORTED, "too many value tokens");
  REQUIRE(p->w_qkv && p->w_o && p->w_val && p->w_off && p->w_attw && p->w_co && p->w_fc1 &&
              p->w_fc2 && p->ln1_beta && p->ln2_beta && p->ln3_beta,
          ILW_E_NULL, "weights and LayerNorm betas must not be NULL");
  REQUIRE(aligned16(p->w_qkv) && aligned16(p->w_o) && aligned16(p->w_val) &&
              aligned16(p->w_off) && aligned16(p->w_attw) && aligned16(p->w_co) &&
              aligned16(p->w_fc1) && aligned16(p->w_fc2),
          ILW_E_PARAM, "weights must be 16-byte aligned");
  const int32_t D = p->dim, NW = p->heads * p->levels * p->points;
  int e;
  if ((e = check_dyadic(p->qkv, 3 * D, "qkv")) || (e = check_dyadic(p->o, D, "o")) ||
      (e = check_dyadic(p->ln1_out, D, "ln1_out")) || (e = check_dyadic(p->val, D, "val")) ||
      (e = check_dyadic(p->off, 2 * NW, "off")) || (e = check_dyadic(p->attw, NW, "attw")) ||
      (e = check_dyadic(p->co, D, "co")) || (e = check_dyadic(p->ln2_out, D, "ln2_out")) ||
      (e = check_dyadic(p->fc1, p->ffn_dim, "fc1")) || (e = check_dyadic(p->fc2, D, "fc2")) ||
      (e = check_dyadic(p->ln3_out, D, "ln3_out")))
    return e;
  if ((e = check_attn(&p->attn))) return e;
  if ((e = check_gelu(p->gelu_I0, p->gelu_k_inter, p->gelu_k_out, p->gelu_mult,
                      p->gelu_shift)))
    return e;
  const int32_t* rm[9] = {&p->res1_mult_a, &p->res1_mult_b, &p->res2_mult_a, &p->res2_mult_b,
                          &p->res3_mult_a, &p->res3_mult_b, &p->res1_shift, &p->res2_shift,
                          &p->res3_shift};
  for (int i = 0; i < 6; ++i)
    if ((e = check_mult(*rm[i], "residual mult"))) return e;
  for (int i = 6; i < 9; ++i)
    if ((e = check_shift(*rm[i], "residual shift"))) return e;
  return ILW_OK;
}

}  // namespace

extern "C" {

const char* ilw_last_error(void) { return g_err.c_str(); }

int ilw_abi_version(void) { return ILW_ABI_VERSION; }

int ilw_linear(const int8_t* x, const int8_t* w, const int32_t* b, ilw_dyadic rq, int8_t* y,
               int64_t M, int32_t N, int32_t K, void* stream) {
  REQUIRE(M >= 0 && N >= 16 && K >= 16, ILW_E_SHAPE, "M=%lld N=%d K=%d invalid",
          (long long)M, N, K);
  REQUIRE(N % 16 == 0 && K % 16 == 0, ILW_E_SHAPE, "N=%d and K=%d must be multiples of 16",
          N, K);
  REQUIRE(K <= 131072, ILW_E_UNSUPPORTED, "K=%d: the int32 accumulator needs K <= 131072",
          K);
  REQUIRE((M + 127) / 128 * ((N + 127) / 128) < (int64_t)1 << 31, ILW_E_UNSUPPORTED,
          "too many tiles");
  if (M == 0) return ok();
  REQUIRE(x && w && y, ILW_E_NULL, "x, w and y must not be NULL");
  REQUIRE(aligned16(x) && aligned16(w) && ((uintptr_t)y & 3) == 0, ILW_E_PARAM,
          "x and w must be 16-byte aligned, y 4-byte aligned");
  int e;
  if ((e = check_dyadic(rq, N, "rq"))) return e;
  GemmArgs a = gemm_args(x, w, b, rq, y, M, N, K);
  return hip_status(launch_gemm(EPI_STORE, a, (hipStream_t)stream), "ilw_linear");
}

int ilw_shiftmax(const int8_t* x, int8_t* y, int64_t rows, int32_t cols, int32_t I0,
                 int32_t k_inter, int32_t k_out, int32_t m_p, int32_t s_d, void* stream) {
  REQUIRE(rows >= 0 && cols >= 1 && cols <= 65536, ILW_E_SHAPE,
          "rows=%lld cols=%d invalid (cols in [1, 65536])", (long long)rows, cols);
  REQUIRE((rows + 3) / 4 < (int64_t)1 << 31, ILW_E_UNSUPPORTED, "too many rows");
  int e;
  if ((e = check_shiftmax(I0, k_inter, k_out, m_p, s_d))) return e;
  if (rows == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  return hip_status(launch_shiftmax(x, y, rows, cols, I0, k_inter, k_out, m_p, s_d,
                                    (hipStream_t)stream),
                    "ilw_shiftmax");
}

int ilw_patch_embed(const int8_t* img, int32_t batch, int32_t channels, int32_t height,
                    int32_t width, int32_t patch, const int8_t* w, const int32_t* bias,
                    ilw_dyadic proj, const int8_t* pos, int32_t pos_mult_a,
                    int32_t pos_mult_b, int32_t pos_shift, int8_t* y, int32_t dim,
                    void* stream) {
  REQUIRE(patch == 16, ILW_E_UNSUPPORTED, "patch = %d: only 16 is implemented", patch);
  REQUIRE(batch >= 0 && channels >= 1 && channels <= 256, ILW_E_SHAPE,
          "batch = %d, channels = %d invalid (channels in [1, 256])", batch, channels);
  REQUIRE(height >= 16 && width >= 16 && height % 16 == 0 && width % 16 == 0, ILW_E_SHAPE,
          "image %dx%d must be a positive multiple of 16 in each side", height, width);
  REQUIRE(dim >= 16 && dim % 16 == 0, ILW_E_SHAPE, "dim = %d must be a multiple of 16", dim);
  const int64_t T = (int64_t)(height / 16) * (width / 16), M = (int64_t)batch * T;
  REQUIRE(M < ((int64_t)1 << 31) && (int64_t)channels * height * width < ((int64_t)1 << 31),
          ILW_E_UNSUPPORTED, "image or token count too large");
  int e;
  if ((e = check_dyadic(proj, dim, "proj"))) return e;
  if ((e = check_mult(pos_mult_a, "pos_mult_a")) || (e = check_mult(pos_mult_b, "pos_mult_b")) ||
      (e = check_shift(pos_shift, "pos_shift")))
    return e;
  if (batch == 0) return ok();
  REQUIRE(img && w && pos && y, ILW_E_NULL, "img, w, pos and y must not be NULL");
  REQUIRE(aligned16(img) && aligned16(w) && ((uintptr_t)pos & 3) == 0 &&
              ((uintptr_t)y & 3) == 0,
          ILW_E_PARAM, "img and w must be 16-byte aligned, pos and y 4-byte aligned");
  GemmArgs a = gemm_args(img, w, bias, proj, y, M, dim, channels * 256);
  a.resid = pos;
  a.res_ma = pos_mult_a;
  a.res_mb = pos_mult_b;
  a.res_shift = pos_shift;
  a.pC = channels;
  a.pH = height;
  a.pW = width;
  a.pgw = width / 16;
  a.pT = (int32_t)T;
  hipStream_t s = (hipStream_t)stream;
  StageTimer t(ILW_STAGE_PATCH_EMBED, s);
  const hipError_t he = launch_gemm(EPI_PATCH, a, s);
  t.done();
  return hip_status(he, "ilw_patch_embed");
}

int ilw_shiftmax_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols, int32_t I0,
                      int32_t k_inter, int32_t k_out, int32_t M, void* stream) {
  REQUIRE(rows >= 0 && cols >= 1 && cols <= 65536, ILW_E_SHAPE,
          "rows=%lld cols=%d invalid (cols in [1, 65536])", (long long)rows, cols);
  REQUIRE((rows + 3) / 4 < (int64_t)1 << 31, ILW_E_UNSUPPORTED, "too many rows");
  int e;
  if ((e = check_shiftmax(I0, k_inter, k_out, 4, 0))) return e;
  REQUIRE(M >= k_out && M <= 32, ILW_E_PARAM, "M = %d must be in [k_out, 32]", M);
  if (rows == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  return hip_status(launch_shiftmax_ivit(x, y, rows, cols, I0, k_inter, k_out, M,
                                         (hipStream_t)stream),
                    "ilw_shiftmax_ivit");
}

int ilw_shiftgelu_ivit(const int8_t* x, int8_t* y, int64_t rows, int32_t cols, int32_t I0,
                       int32_t k_inter, int32_t k_out, int32_t out_mult, int32_t out_shift,
                       void* stream) {
  REQUIRE(rows >= 0 && cols >= 1 && cols <= 65536, ILW_E_SHAPE,
          "rows=%lld cols=%d invalid (cols in [1, 65536])", (long long)rows, cols);
  REQUIRE((rows + 3) / 4 < (int64_t)1 << 31, ILW_E_UNSUPPORTED, "too many rows");
  int e;
  if ((e = check_gelu(I0, k_inter, k_out, out_mult, out_shift))) return e;
  if (rows == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  return hip_status(launch_shiftgelu_ivit(x, y, rows, cols, I0, k_inter, k_out, out_mult,
                                          out_shift, (hipStream_t)stream),
                    "ilw_shiftgelu_ivit");
}

int ilw_sdshiftgelu(const int8_t* x, int8_t* y, int64_t n, int32_t I0, int32_t k_inter,
                    int32_t k_out, int32_t out_mult, int32_t out_shift, void* stream) {
  REQUIRE(n >= 0, ILW_E_SHAPE, "n=%lld must be >= 0", (long long)n);
  int e;
  if ((e = check_gelu(I0, k_inter, k_out, out_mult, out_shift))) return e;
  if (n == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  REQUIRE(aligned16(x) && aligned16(y), ILW_E_PARAM, "x and y must be 16-byte aligned");
  return hip_status(launch_gelu(x, y, n, I0, k_inter, k_out, out_mult, out_shift,
                                (hipStream_t)stream),
                    "ilw_sdshiftgelu");
}

int ilw_int_layernorm(const int8_t* x, int8_t* y, int64_t rows, int32_t C,
                      const int32_t* beta, ilw_dyadic out, int32_t newton_iters,
                      void* stream) {
  REQUIRE(rows >= 0 && C >= 4 && C <= 16384 && C % 4 == 0, ILW_E_SHAPE,
          "rows=%lld C=%d invalid (C a multiple of 4 in [4, 16384])", (long long)rows, C);
  REQUIRE(newton_iters >= 1 && newton_iters <= 64, ILW_E_PARAM,
          "newton_iters = %d must be in [1, 64]", newton_iters);
  REQUIRE((rows + 3) / 4 < (int64_t)1 << 31, ILW_E_UNSUPPORTED, "too many rows");
  int e;
  if ((e = check_dyadic(out, C, "out"))) return e;
  if (rows == 0) return ok();
  REQUIRE(x && y && beta, ILW_E_NULL, "x, y and beta must not be NULL");
  REQUIRE(((uintptr_t)x & 3) == 0 && ((uintptr_t)y & 3) == 0, ILW_E_PARAM,
          "x and y must be 4-byte aligned");
  return hip_status(launch_layernorm(x, y, rows, C, beta, out.mult, out.shift, out.n,
                                     newton_iters, (hipStream_t)stream),
                    "ilw_int_layernorm");
}

int ilw_residual_add(const int8_t* a, const int8_t* b, int8_t* y, int64_t n, int32_t mult_a,
                     int32_t mult_b, int32_t shift, void* stream) {
  REQUIRE(n >= 0, ILW_E_SHAPE, "n=%lld must be >= 0", (long long)n);
  int e;
  if ((e = check_mult(mult_a, "mult_a")) || (e = check_mult(mult_b, "mult_b")) ||
      (e = check_shift(shift, "shift")))
    return e;
  if (n == 0) return ok();
  REQUIRE(a && b && y, ILW_E_NULL, "a, b and y must not be NULL");
  REQUIRE(aligned16(a) && aligned16(b) && aligned16(y), ILW_E_PARAM,
          "a, b and y must be 16-byte aligned");
  return hip_status(launch_residual(a, b, y, n, mult_a, mult_b, shift, (hipStream_t)stream),
                    "ilw_residual_add");
}

size_t ilw_attention_workspace_bytes(int32_t batch, int32_t grid_h, int32_t grid_w,
                                     int32_t win_h, int32_t win_w, int32_t dim,
                                     int32_t head_dim) {
  Geometry g;
  if (check_geometry(batch, grid_h, grid_w, win_h, win_w, &g)) return 0;
  if ((head_dim != 32 && head_dim != 64) || dim < head_dim || dim % head_dim) {
    fail(ILW_E_SHAPE, "dim = %d must be a positive multiple of head_dim = %d (32 or 64)", dim,
         head_dim);
    return 0;
  }
  ok();
  return qkv_bytes(batch, g, dim, nullptr, nullptr, head_dim);
}

int ilw_attention(const int8_t* qkv, int8_t* out, int32_t batch, int32_t grid_h,
                  int32_t grid_w, int32_t win_h, int32_t win_w, int32_t dim, int32_t heads,
                  int32_t head_dim, const ilw_attn_params* ap, void* workspace,
                  size_t workspace_bytes, void* stream) {
  REQUIRE(head_dim == 32 || head_dim == 64, ILW_E_UNSUPPORTED,
          "head_dim = %d: 32 and 64 are implemented", head_dim);
  REQUIRE(heads >= 1 && dim == heads * head_dim, ILW_E_SHAPE,
          "dim = %d must equal heads (%d) * head_dim", dim, heads);
  Geometry g;
  int e;
  if ((e = check_geometry(batch, grid_h, grid_w, win_h, win_w, &g))) return e;
  if ((e = check_attn(ap))) return e;
  if (batch == 0) return ok();
  REQUIRE(qkv && out, ILW_E_NULL, "qkv and out must not be NULL");
  REQUIRE(aligned16(qkv) && aligned16(out), ILW_E_PARAM,
          "qkv and out must be 16-byte aligned");
  const size_t need = qkv_bytes(batch, g, dim, nullptr, nullptr, head_dim);
  REQUIRE(workspace && workspace_bytes >= need, ILW_E_WORKSPACE,
          "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  REQUIRE(aligned16(workspace), ILW_E_PARAM, "workspace must be 16-byte aligned");
  QkvLayout L;
  qkv_bytes(batch, g, dim, &L, (int8_t*)workspace, head_dim);
  hipStream_t s = (hipStream_t)stream;
  hipError_t he;
  {
    StageTimer t(ILW_STAGE_RELAYOUT, s);
    he = launch_qkv_relayout(qkv, batch, L, s);
    t.done();
  }
  if (he == hipSuccess) {
    StageTimer t(ILW_STAGE_ATTENTION, s);
    he = launch_attention(attn_args(L, out, batch, *ap), s);
    t.done();
  }
  return hip_status(he, "ilw_attention");
}

size_t ilw_block_workspace_bytes(const ilw_block_params* p, int32_t batch, int32_t grid_h,
                                 int32_t grid_w, int32_t win_h, int32_t win_w) {
  Geometry g;
  if (check_block(p, batch, grid_h, grid_w, win_h, win_w, &g)) return 0;
  ok();
  return block_layout(p, batch, g, nullptr, nullptr);
}

int ilw_block_forward(const ilw_block_params* p, const int8_t* x, int8_t* y, int32_t batch,
                      int32_t grid_h, int32_t grid_w, int32_t win_h, int32_t win_w,
                      void* workspace, size_t workspace_bytes, void* stream) {
  Geometry g;
  int e;
  if ((e = check_block(p, batch, grid_h, grid_w, win_h, win_w, &g))) return e;
  if (batch == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  REQUIRE(aligned16(x) && aligned16(y), ILW_E_PARAM, "x and y must be 16-byte aligned");
  const size_t need = block_layout(p, batch, g, nullptr, nullptr);
  REQUIRE(workspace && workspace_bytes >= need, ILW_E_WORKSPACE,
          "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  REQUIRE(aligned16(workspace), ILW_E_PARAM, "workspace must be 16-byte aligned");
  BlockLayout L;
  block_layout(p, batch, g, (int8_t*)workspace, &L);
  hipError_t he = pack_block_weights(&p, &L, 1, (hipStream_t)stream);
  if (he != hipSuccess) return hip_status(he, "ilw_block_forward weight packing");
  int ready = READY_NONE;
  return run_block(p, nullptr, nullptr, x, y, batch, g, L, READY_NONE, &ready,
                   (hipStream_t)stream);
}

int ilw_block_forward_noalloc(const ilw_block_params* p, const int8_t* x, int8_t* y,
                              int32_t batch, int32_t grid_h, int32_t grid_w, int32_t win_h,
                              int32_t win_w, void* stream) {
  Geometry g;
  int e;
  if ((e = check_block(p, batch, grid_h, grid_w, win_h, win_w, &g))) return e;
  if (batch == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  REQUIRE(aligned16(x) && aligned16(y), ILW_E_PARAM, "x and y must be 16-byte aligned");
  const size_t need = block_layout(p, batch, g, nullptr, nullptr);
  REQUIRE(need <= ILW_NOALLOC_SCRATCH_BYTES, ILW_E_WORKSPACE,
          "ilw_block_forward_noalloc: this block needs %zu bytes of scratch, above the "
          "static scratch of %zu bytes (use ilw_block_forward with a workspace)",
          need, (size_t)ILW_NOALLOC_SCRATCH_BYTES);
  int8_t* ws = nullptr;
  if ((e = scratch_of_current_device(&ws))) return e;
  BlockLayout L;
  block_layout(p, batch, g, ws, &L);
  hipError_t he = pack_block_weights(&p, &L, 1, (hipStream_t)stream);
  if (he != hipSuccess) return hip_status(he, "ilw_block_forward_noalloc weight packing");
  int ready = READY_NONE;
  return run_block(p, nullptr, nullptr, x, y, batch, g, L, READY_NONE, &ready,
                   (hipStream_t)stream);
}

size_t ilw_encoder_workspace_bytes(const ilw_block_params* blocks, int32_t n_blocks,
                                   const int32_t* windows, int32_t batch, int32_t grid_h,
                                   int32_t grid_w) {
  if (check_encoder(blocks, n_blocks, windows, batch, grid_h, grid_w)) return 0;
  ok();
  return encoder_workspace(blocks, n_blocks, windows, batch, grid_h, grid_w);
}

int ilw_encoder_forward(const ilw_block_params* blocks, int32_t n_blocks,
                        const int32_t* windows, const int8_t* x, int8_t* y, int32_t batch,
                        int32_t grid_h, int32_t grid_w, void* workspace,
                        size_t workspace_bytes, void* stream) {
  int e;
  if ((e = check_encoder(blocks, n_blocks, windows, batch, grid_h, grid_w))) return e;
  if (batch == 0) return ok();
  REQUIRE(x && y, ILW_E_NULL, "x and y must not be NULL");
  REQUIRE(aligned16(x) && aligned16(y), ILW_E_PARAM, "x and y must be 16-byte aligned");
  const size_t need = encoder_workspace(blocks, n_blocks, windows, batch, grid_h, grid_w);
  REQUIRE(workspace && workspace_bytes >= need, ILW_E_WORKSPACE,
          "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  REQUIRE(aligned16(workspace), ILW_E_PARAM, "workspace must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  // Block b reads its input from x (b = 0) or y and writes y.  The workspace
  // regions h and Q K V^T sit at the same offsets for every block, so block
  // b can leave block b + 1's LN1 output (fused fc2 epilogue) or its Q, K,
  // V^T (block tail kernel) there.
  const size_t qres = encoder_qkv_reserve(blocks, n_blocks, windows, batch, grid_h, grid_w);
  // the 384-channel LayerNorm-fused linears read their weights packed in
  // MFMA fragment order: every block's are packed first, in one launch
  const size_t shared = encoder_shared_bytes(blocks, n_blocks, windows, batch, grid_h, grid_w);
  std::vector<BlockLayout> Ls((size_t)n_blocks);
  std::vector<const ilw_block_params*> ps((size_t)n_blocks);
  {
    size_t off = shared;
    for (int32_t b = 0; b < n_blocks; ++b) {
      Geometry g;
      check_geometry(batch, grid_h, grid_w, windows[2 * b], windows[2 * b + 1], &g);
      block_layout(&blocks[b], batch, g, (int8_t*)workspace, &Ls[b], qres, false);
      off += packed_layout(&blocks[b], (int64_t)batch * g.T, (int8_t*)workspace, off, &Ls[b]);
      ps[b] = &blocks[b];
    }
    const hipError_t he = pack_block_weights(ps.data(), Ls.data(), n_blocks, s);
    if (he != hipSuccess) return hip_status(he, "ilw_encoder_forward weight packing");
  }
  int ready = READY_NONE;
  for (int32_t b = 0; b < n_blocks; ++b) {
    Geometry g;
    check_geometry(batch, grid_h, grid_w, windows[2 * b], windows[2 * b + 1], &g);
    const BlockLayout& L = Ls[b];
    const ilw_block_params* next = b + 1 < n_blocks ? &blocks[b + 1] : nullptr;
    QkvLayout nq;
    if (next) nq = Ls[b + 1].qkv;
    int ready_out = READY_NONE;
    if ((e = run_block(&blocks[b], next, next ? &nq : nullptr, b == 0 ? x : y, y, batch, g, L,
                       ready, &ready_out, s)))
      return e;
    ready = ready_out;
  }
  return ok();
}

int ilw_split_conv(int32_t n_branches, const int8_t* const* x, const int32_t* channels,
                   const int8_t* const* w, const ilw_dyadic* branch, const int32_t* bias,
                   ilw_dyadic out, int8_t* y, int64_t M, int32_t N, void* stream) {
  REQUIRE(n_branches >= 1 && n_branches <= kMaxBranches, ILW_E_SHAPE,
          "n_branches = %d must be in [1, %d]", n_branches, kMaxBranches);
  REQUIRE(x && channels && w && branch, ILW_E_NULL,
          "x, channels, w and branch (host arrays) must not be NULL");
  REQUIRE(M >= 0 && N >= 16 && N % 16 == 0, ILW_E_SHAPE,
          "M = %lld, N = %d invalid (N a positive multiple of 16)", (long long)M, N);
  REQUIRE((M + 63) / 64 * ((N + 63) / 64) < (int64_t)1 << 31, ILW_E_UNSUPPORTED,
          "too many tiles");
  int e;
  SplitArgs a = {};
  a.nbr = n_branches;
  int32_t ks = 0;
  for (int32_t b = 0; b < n_branches; ++b) {
    REQUIRE(channels[b] >= 64 && channels[b] <= 65536 && channels[b] % 64 == 0, ILW_E_SHAPE,
            "channels[%d] = %d must be a multiple of 64 in [64, 65536]", b, channels[b]);
    if ((e = check_dyadic(branch[b], N, "branch"))) return e;
    a.C[b] = channels[b];
    a.kstart[b] = ks;
    ks += channels[b] / 64;
    a.bmult[b] = branch[b].mult;
    a.bshift[b] = branch[b].shift;
    a.bnq[b] = branch[b].n;
  }
  a.kstart[n_branches] = ks;
  if ((e = check_dyadic(out, N, "out"))) return e;
  if (M == 0) return ok();
  REQUIRE(y, ILW_E_NULL, "y must not be NULL");
  REQUIRE(((uintptr_t)y & 3) == 0, ILW_E_PARAM, "y must be 4-byte aligned");
  for (int32_t b = 0; b < n_branches; ++b) {
    REQUIRE(x[b] && w[b], ILW_E_NULL, "x[%d] and w[%d] must not be NULL", b, b);
    REQUIRE(aligned16(x[b]) && aligned16(w[b]), ILW_E_PARAM,
            "x[%d] and w[%d] must be 16-byte aligned", b, b);
    a.x[b] = x[b];
    a.w[b] = w[b];
  }
  a.bias = bias;
  a.omult = out.mult;
  a.oshift = out.shift;
  a.onq = out.n;
  a.y = y;
  a.M = M;
  a.N = N;
  hipStream_t s = (hipStream_t)stream;
  StageTimer t(ILW_STAGE_SPLIT_CONV, s);
  const hipError_t he = launch_split_conv(a, s);
  t.done();
  return hip_status(he, "ilw_split_conv");
}

namespace {
// offsets: int16 Q8, or (offsets8 set) int8 values used as offsets8 << off_shift
int deform_impl(const int8_t* value, const int32_t* level_hw, const int32_t* level_start,
                int32_t L, int32_t P, const int32_t* ref, int32_t ref_dims,
                const int16_t* offsets, const int8_t* logits, int8_t* out, int32_t B, int32_t Q,
                int32_t heads, int32_t head_dim, int32_t I0, int32_t k_inter, int32_t k_out,
                int32_t m_p, int32_t s_d, int32_t out_mult, int32_t out_shift, int32_t mode,
                void* stream, const char* name,
                const int8_t* offsets8 = nullptr, int32_t off_shift = 0) {
  REQUIRE(level_hw && level_start, ILW_E_NULL, "level_hw and level_start (host) required");
  REQUIRE(ref_dims == 2 || ref_dims == 4, ILW_E_PARAM,
          "ref_dims = %d: references are points (2) or boxes (4)", ref_dims);
  REQUIRE(L >= 1 && L <= kMaxLevels && P >= 1 && L * P <= 64, ILW_E_SHAPE,
          "L=%d P=%d invalid (L in [1, 8], L*P in [1, 64])", L, P);
  REQUIRE(B >= 0 && Q >= 0 && heads >= 1, ILW_E_SHAPE, "B=%d Q=%d heads=%d invalid", B, Q,
          heads);
  REQUIRE(head_dim >= 4 && head_dim <= 256 && head_dim % 4 == 0, ILW_E_SHAPE,
          "head_dim = %d must be a multiple of 4 in [4, 256]", head_dim);
  REQUIRE(mode == 0 || mode == 1, ILW_E_PARAM, "mode = %d must be 0 or 1", mode);
  int e;
  if ((e = check_shiftmax(I0, k_inter, k_out, m_p, s_d))) return e;
  if ((e = check_mult(out_mult, "out_mult"))) return e;
  REQUIRE(out_shift >= 1 && out_shift <= (mode == 0 ? 62 : 46), ILW_E_PARAM,
          "out_shift = %d out of range for mode %d", out_shift, mode);
  DeformArgs a = {};
  int64_t S = 0;
  for (int32_t l = 0; l < L; ++l) {
    const int32_t hl = level_hw[2 * l], wl = level_hw[2 * l + 1];
    REQUIRE(hl >= 1 && hl <= 32767 && wl >= 1 && wl <= 32767, ILW_E_SHAPE,
            "level %d size %dx%d invalid", l, hl, wl);
    REQUIRE(level_start[l] >= 0, ILW_E_SHAPE, "level_start[%d] < 0", l);
    a.hw[l][0] = hl;
    a.hw[l][1] = wl;
    a.start[l] = level_start[l];
    const int64_t end = (int64_t)level_start[l] + (int64_t)hl * wl;
    S = end > S ? end : S;
  }
  REQUIRE(S <= INT32_MAX, ILW_E_SHAPE, "value rows exceed int32");
  const int64_t groups = (int64_t)B * Q * heads;
  REQUIRE((groups * (head_dim / 4) + 255) / 256 < (int64_t)1 << 31, ILW_E_UNSUPPORTED,
          "too many queries");
  if (groups == 0) return ok();
  REQUIRE(value && ref && (offsets || offsets8) && logits && out, ILW_E_NULL,
          "value, ref, offsets, logits and out must not be NULL");
  REQUIRE(((uintptr_t)value & 3) == 0 && ((uintptr_t)out & 3) == 0, ILW_E_PARAM,
          "value and out must be 4-byte aligned");
  a.value = value;
  a.ref = ref;
  a.offs = offsets;
  a.logits = logits;
  a.out = out;
  a.B = B;
  a.Q = Q;
  a.H = heads;
  a.Dh = head_dim;
  a.L = L;
  a.P = P;
  a.S = (int32_t)S;
  a.I0 = I0;
  a.k_inter = k_inter;
  a.k_out = k_out;
  a.m_p = m_p;
  a.s_d = s_d;
  a.out_mult = out_mult;
  a.out_shift = out_shift;
  a.mode = mode;
  a.ref_dims = ref_dims;
  a.offs8 = offsets8;
  a.off_shift = off_shift;
  StageTimer t(ILW_STAGE_DEFORM, (hipStream_t)stream);
  hipError_t he = launch_deform(a, (hipStream_t)stream);
  t.done();
  return hip_status(he, name);
}
}  // namespace

int ilw_deform_attn(const int8_t* value, const int32_t* level_hw, const int32_t* level_start,
                    int32_t L, int32_t P, const int32_t* ref, const int16_t* offsets,
                    const int8_t* logits, int8_t* out, int32_t B, int32_t Q, int32_t heads,
                    int32_t head_dim, int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p,
                    int32_t s_d, int32_t out_mult, int32_t out_shift, int32_t mode,
                    void* stream) {
  return deform_impl(value, level_hw, level_start, L, P, ref, 2, offsets, logits, out, B, Q,
                     heads, head_dim, I0, k_inter, k_out, m_p, s_d, out_mult, out_shift, mode,
                     stream, "ilw_deform_attn");
}

int ilw_deform_attn_boxes(const int8_t* value, const int32_t* level_hw,
                          const int32_t* level_start, int32_t L, int32_t P,
                          const int32_t* ref, const int16_t* offsets, const int8_t* logits,
                          int8_t* out, int32_t B, int32_t Q, int32_t heads, int32_t head_dim,
                          int32_t I0, int32_t k_inter, int32_t k_out, int32_t m_p, int32_t s_d,
                          int32_t out_mult, int32_t out_shift, int32_t mode, void* stream) {
  return deform_impl(value, level_hw, level_start, L, P, ref, 4, offsets, logits, out, B, Q,
                     heads, head_dim, I0, k_inter, k_out, m_p, s_d, out_mult, out_shift, mode,
                     stream, "ilw_deform_attn_boxes");
}

size_t ilw_decoder_workspace_bytes(const ilw_decoder_params* p, int32_t batch,
                                   int32_t queries, int32_t value_tokens) {
  if (check_decoder(p, batch, queries, value_tokens)) return 0;
  ok();
  return decoder_layout(p, batch, queries, value_tokens, nullptr, nullptr);
}

int ilw_decoder_layer(const ilw_decoder_params* p, const int8_t* tgt, const int8_t* memory,
                      const int32_t* ref, const int32_t* level_hw, const int32_t* level_start,
                      int8_t* y, int32_t batch, int32_t queries, int32_t value_tokens,
                      void* workspace, size_t workspace_bytes, void* stream) {
  int e;
  if ((e = check_decoder(p, batch, queries, value_tokens))) return e;
  if (batch == 0) return ok();
  REQUIRE(tgt && memory && ref && y && level_hw && level_start, ILW_E_NULL,
          "tgt, memory, ref, y, level_hw and level_start must not be NULL");
  REQUIRE(aligned16(tgt) && aligned16(memory) && aligned16(y), ILW_E_PARAM,
          "tgt, memory and y must be 16-byte aligned");
  REQUIRE(y != tgt, ILW_E_PARAM, "y must not alias tgt");
  const size_t need = decoder_layout(p, batch, queries, value_tokens, nullptr, nullptr);
  REQUIRE(workspace && workspace_bytes >= need, ILW_E_WORKSPACE,
          "workspace of %zu bytes needed, %zu given", need, workspace_bytes);
  REQUIRE(aligned16(workspace), ILW_E_PARAM, "workspace must be 16-byte aligned");
  DecoderLayout L;
  decoder_layout(p, batch, queries, value_tokens, (int8_t*)workspace, &L);
  hipStream_t s = (hipStream_t)stream;
  const int32_t D = p->dim, H = p->heads, hd = D / H, F = p->ffn_dim;
  const int32_t NW = H * p->levels * p->points, NO = 2 * NW;
  const int64_t MQ = (int64_t)batch * queries, MS = (int64_t)batch * value_tokens;
  hipError_t he = hipSuccess;
  auto run = [&](int stage, auto&& launch) {
    if (he != hipSuccess) return;
    StageTimer t(stage, s);
    he = launch();
    t.done();
  };
  auto ln = [&](const int8_t* in, int8_t* out, const int32_t* beta, const ilw_dyadic& d) {
    run(ILW_STAGE_LAYERNORM, [&] {
      return launch_layernorm(in, out, MQ, D, beta, d.mult, d.shift, d.n, p->ln_iters, s);
    });
  };
  auto resid = [&](GemmArgs a, const int8_t* skip, int32_t ma, int32_t mb, int32_t sh) {
    a.resid = skip;
    a.res_ma = ma;
    a.res_mb = mb;
    a.res_shift = sh;
    run(ILW_STAGE_DECODER, [&] { return launch_gemm(EPI_RESID, a, s); });
  };
  auto plain = [&](const GemmArgs& a) {
    run(ILW_STAGE_DECODER, [&] { return launch_gemm(EPI_STORE, a, s); });
  };
  // residual add and post-norm LayerNorm: one GEMM with the LayerNorm in its
  // epilogue where the tile can hold whole rows, else GEMM then LayerNorm
  const bool fuse = ln_fusable(D);
  auto resid_ln = [&](GemmArgs a, const int8_t* skip, int32_t ma, int32_t mb, int32_t sh,
                      const int32_t* beta, const ilw_dyadic& d, int8_t* out) {
    if (!fuse) {
      resid(a, skip, ma, mb, sh);
      ln(a.y, out, beta, d);
      return;
    }
    a.resid = skip;
    a.res_ma = ma;
    a.res_mb = mb;
    a.res_shift = sh;
    run(ILW_STAGE_DECODER,
        [&] { return launch_gemm(EPI_RESID_LN, with_ln(a, beta, d, p->ln_iters, out), s); });
  };

  // self-attention over the queries (one global window per image)
  GemmArgs a = gemm_args(tgt, p->w_qkv, p->b_qkv, p->qkv, nullptr, MQ, 3 * D, D);
  a.qkv = L.qkv;
  run(ILW_STAGE_GEMM_QKV, [&] { return launch_gemm(EPI_QKV, a, s); });
  run(ILW_STAGE_ATTENTION, [&] { return launch_attention(attn_args(L.qkv, L.att, batch, p->attn), s); });
  resid_ln(gemm_args(L.att, p->w_o, p->b_o, p->o, L.x, MQ, D, D), tgt, p->res1_mult_a,
           p->res1_mult_b, p->res1_shift, p->ln1_beta, p->ln1_out, L.t1);
  // cross-attention: value projection, offsets (int8 1/16 px -> Q8), weights
  plain(gemm_args(memory, p->w_val, p->b_val, p->val, L.v, MS, D, D));
  plain(gemm_args(L.t1, p->w_off, p->b_off, p->off, L.off8, MQ, NO, D));
  plain(gemm_args(L.t1, p->w_attw, p->b_attw, p->attw, L.lg, MQ, NW, D));
  if (he != hipSuccess) return hip_status(he, "ilw_decoder_layer");
  // the sampler reads the int8 offsets (1/16 px) and widens them to Q8 itself
  if ((e = deform_impl(L.v, level_hw, level_start, p->levels, p->points, ref, p->ref_dims,
                       nullptr, L.lg, L.smp, batch, queries, H, hd, p->da_I0, 16, 8, 4,
                       p->da_s_d, p->da_out_mult, p->da_out_shift, p->da_mode, stream,
                       "ilw_decoder_layer sampler", L.off8, 4)))
    return e;
  resid_ln(gemm_args(L.smp, p->w_co, p->b_co, p->co, L.x, MQ, D, D), L.t1, p->res2_mult_a,
           p->res2_mult_b, p->res2_shift, p->ln2_beta, p->ln2_out, L.t2);
  // FFN
  a = gemm_args(L.t2, p->w_fc1, p->b_fc1, p->fc1, L.g, MQ, F, D);
  a.g_I0 = p->gelu_I0;
  a.g_kinter = p->gelu_k_inter;
  a.g_kout = p->gelu_k_out;
  a.g_mult = p->gelu_mult;
  a.g_shift = p->gelu_shift;
  run(ILW_STAGE_DECODER, [&] { return launch_gemm(EPI_GELU, a, s); });
  resid_ln(gemm_args(L.g, p->w_fc2, p->b_fc2, p->fc2, L.x, MQ, D, F), L.t2, p->res3_mult_a,
           p->res3_mult_b, p->res3_shift, p->ln3_beta, p->ln3_out, y);
  return hip_status(he, "ilw_decoder_layer");
}

int ilw_profile_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on.store(enable != 0);
  g_prof.recs.clear();
  g_prof.used = 0;
  return ok();
}

int ilw_profile_read(double* total_ms, int32_t* launches, int32_t n_stages) {
  REQUIRE(total_ms && launches, ILW_E_NULL, "output arrays must not be NULL");
  REQUIRE(n_stages >= 0, ILW_E_SHAPE, "n_stages < 0");
  std::lock_guard<std::mutex> lk(g_prof.mu);
  for (int32_t i = 0; i < n_stages; ++i) {
    total_ms[i] = 0.0;
    launches[i] = 0;
  }
  if (!g_prof.recs.empty()) {
    hipError_t e = hipEventSynchronize(g_prof.recs.back().stop);
    if (e != hipSuccess) return hip_status(e, "ilw_profile_read");
  }
  for (const ProfRecord& r : g_prof.recs) {
    if (r.stage >= n_stages) continue;
    float ms = 0.f;
    hipError_t e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return hip_status(e, "ilw_profile_read");
    total_ms[r.stage] += ms;
    launches[r.stage] += 1;
  }
  return ok();
}

}  // extern "C"
