// C ABI of the SSD verify-step library: model upload, sessions, the verify
// step and the image schedule driver.  See include/ssd.h for the contract.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <chrono>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "ssd_internal.h"

using namespace ssd;

namespace {

thread_local std::string g_err;

// per-round accept counters of an image decode: the (j+1)-th verify round of a
// block counts under j (rounds past the last counted under NCNT_ROUNDS - 1)
constexpr int NCNT_ROUNDS = 8;

ssd_status fail(ssd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

struct HipError {
  hipError_t e;
  const char* what;
};

#define HIPCHK(x)                                 \
  do {                                            \
    hipError_t e_ = (x);                          \
    if (e_ != hipSuccess) throw HipError{e_, #x}; \
  } while (0)

// host or device pointer?
bool is_device_ptr(const void* p) {
  if (!p) return false;
  hipPointerAttribute_t attr;
  hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged;
}

struct Allocs {
  std::vector<void*> ptrs;
  ~Allocs() {
    for (void* p : ptrs) (void)hipFree(p);
  }
  template <typename T>
  T* get(size_t count) {
    void* p = nullptr;
    size_t bytes = count * sizeof(T);
    if (bytes == 0) bytes = 16;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      throw HipError{e, "hipMalloc"};
    }
    ptrs.push_back(p);
    return (T*)p;
  }
};

int64_t numel_of(const ssd_model_config& c) {
  const int64_t d = c.d_model, D = c.head_dim, f = c.d_ff;
  int64_t per_layer = d + (int64_t)c.n_heads * D * d + 2LL * c.n_kv_heads * D * d + d * (int64_t)c.n_heads * D + d +
                      2 * f * d + d * f;
  return (int64_t)c.vocab * d * 2 + d + per_layer * c.n_layers;
}

ssd_status validate_config(const ssd_model_config* c) {
  if (!c) return fail(SSD_E_INVAL, "config is NULL");
  if (c->n_layers < 1 || c->d_model < 2 || c->n_heads < 1 || c->n_kv_heads < 1 || c->head_dim < 2 || c->d_ff < 1 ||
      c->vocab < 1)
    return fail(SSD_E_INVAL, "non-positive model dimension");
  if (c->n_heads % c->n_kv_heads) return fail(SSD_E_INVAL, "n_heads must be a multiple of n_kv_heads");
  if (c->head_dim % 2) return fail(SSD_E_INVAL, "head_dim must be even");
  if (c->img_lo < 0 || c->img_hi > c->vocab || c->img_hi - c->img_lo < 2)
    return fail(SSD_E_INVAL, "image range [%d,%d) invalid for vocab %d", c->img_lo, c->img_hi, c->vocab);
  if (c->dtype != SSD_F32 && c->dtype != SSD_BF16) return fail(SSD_E_INVAL, "unknown dtype");
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 0.f)) return fail(SSD_E_INVAL, "rms_eps and rope_theta must be > 0");
  if (c->dtype == SSD_BF16) {
    if (c->d_model % 256 || (c->n_heads * c->head_dim) % 256 || c->d_ff % 256)
      return fail(SSD_E_INVAL, "bf16 models need d_model, n_heads*head_dim and d_ff multiples of 256");
    if (c->head_dim != 128 && c->head_dim != 64) return fail(SSD_E_INVAL, "bf16 models need head_dim 64 or 128");
    if (c->d_model > 64 * GEMM_RMS_MAX_PARTS) return fail(SSD_E_INVAL, "bf16 models need d_model <= %d", 64 * GEMM_RMS_MAX_PARTS);
    if ((c->img_hi - c->img_lo) % 16) return fail(SSD_E_INVAL, "bf16 models need an image range multiple of 16");
  } else {
    if ((c->img_hi - c->img_lo) % 2 || c->d_model % 2) return fail(SSD_E_INVAL, "fp32 models need even d_model and image range");
  }
  return SSD_OK;
}

}  // namespace

struct ssd_session;

namespace ssd {
thread_local LaunchTimer* g_launch_timer = nullptr;
}

namespace {
// Per-launch timing of kernel classes (measurement hook): the GEMM and
// attention launches of a class run with dispatch-timestamp events.
struct Prof : LaunchTimer {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  struct Mark {
    int cls;
    hipEvent_t a, b;
    double bytes, flops;
    bool tiled;
  };
  std::vector<Mark> marks;
  // qkv, o, gate_up, down, lm_head, attention, persistent forward; then the
  // launches of classes 0-4 that ran on the tiled GEMM kernel, counted again
  static constexpr int NCLS = 8;
  static constexpr int TILED = 7;
  double ms[NCLS] = {}, bytes[NCLS] = {}, flops[NCLS] = {};
  int64_t n[NCLS] = {};
  int cur_cls = 0;
  double cur_bytes = 0, cur_flops = 0;
  bool cur_tiled = false;
  hipEvent_t get() {
    if (used == pool.size()) {
      hipEvent_t e;
      HIPCHK(hipEventCreate(&e));
      pool.push_back(e);
    }
    return pool[used++];
  }
  void next(hipEvent_t& a, hipEvent_t& b) override {
    a = get();
    b = get();
    marks.push_back(Mark{cur_cls, a, b, cur_bytes, cur_flops, cur_tiled});
    cur_bytes = 0;  // a call's algorithmic bytes and flops go with its first launch
    cur_flops = 0;
  }
  // time the launches of one call of class cls (b algorithmic bytes, fl
  // algorithmic flops; tiled: a GEMM on the tiled kernel)
  template <typename F>
  void run(int cls, double b, hipStream_t st, F&& f, double fl = 0.0, bool tiled = false) {
    (void)st;
    if (!on) {
      f();
      return;
    }
    cur_cls = cls;
    cur_bytes = b;
    cur_flops = fl;
    cur_tiled = tiled;
    g_launch_timer = this;
    try {
      f();
    } catch (...) {
      g_launch_timer = nullptr;
      throw;
    }
    g_launch_timer = nullptr;
  }
  // after the stream has drained
  void flush() {
    for (const Mark& m : marks) {
      float t = 0.f;
      HIPCHK(hipEventSynchronize(m.b));  // launches may sit on a session's own stream
      HIPCHK(hipEventElapsedTime(&t, m.a, m.b));
      ms[m.cls] += t;
      bytes[m.cls] += m.bytes;
      flops[m.cls] += m.flops;
      n[m.cls] += 1;
      if (m.tiled) {
        ms[TILED] += t;
        bytes[TILED] += m.bytes;
        flops[TILED] += m.flops;
        n[TILED] += 1;
      }
    }
    marks.clear();
    used = 0;
  }
  ~Prof() override {
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }
};
}  // namespace

namespace {

// Workspace of the allocation-free draft-head run (ssd_draft_head_run_noalloc):
// a static device array, one copy on every GPU the library runs on, held until
// the process ends.  Host code never passes `scratch` itself to a kernel or a
// copy: the host-side name only stands in for the symbol; the device address
// comes from hipGetSymbolAddress, looked up once per device.
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};
bool g_scratch_done[MAX_DEVICES] = {};

// The current device's copy of `scratch` (nullptr if its address is unknown);
// the first call on a device looks it up with that device current.
void* scratch_of_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_done[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess && p != nullptr) {
      g_scratch_ptr[dev] = p;
    } else {
      (void)hipGetLastError();
      g_scratch_ptr[dev] = nullptr;
    }
    g_scratch_done[dev] = true;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

struct ssd_model {
  ssd_model_config cfg;
  Dims dm;
  hipStream_t stream;
  Allocs mem;
  void* emb = nullptr;
  std::vector<LayerW> layers;
  float* gf = nullptr;
  void* wlm = nullptr;
  bool poisoned = false;
  ssd_session* dec = nullptr;  // cached decode workspace
  int dec_B = 0, dec_P = 0, dec_L = 0, dec_K = 0;
  int xcd = 0;  // XCD count when workgroups are dispatched round-robin over XCDs (see xcd_grid), else 0
  // persistent forward pass (index MT - 1: one or two 16-token tiles): grid
  // size (0: not available) and its XCD mapping (0: fenced reductions)
  int fwd_grid[2] = {0, 0};
  int fwd_xcd[2] = {0, 0};
  unsigned fwd_spin_limit = 0;  // polls before a dependency wait of the persistent pass gives up
  Prof prof;
  void* scratch = nullptr;  // this model's device's copy of the static workspace (allocation-free runs)
};

struct ssd_session {
  ssd_model* m;
  Dims dm;
  hipStream_t stream;
  int B, P, Lmax, Kmax, Mmax, ring;
  int max_ctx;         // the caller's bound on P + committed and drafted positions (Lmax rounds it up)
  std::vector<int> f;  // host mirror of the frontier
  bool poisoned = false;
  Allocs mem;
  int* d_f;
  int* tok;         // [Mmax] working token ids
  unsigned char* acc;
  int* cnt;
  int* amax;
  float* x;
  void* xn;
  float* ssq;
  int ssq_rows_ld;
  size_t xn_plane, q_plane, o_plane, h_plane;  // lo-plane offsets (elements) of the split activations
  void* q;
  void* o;
  void* h;
  float* logits;
  float* carry;
  float* ref;
  float* refstage;  // device copy of caller-provided reference logits [B][Kmax][V_img]
  int* ref_flag;
  void* kc;
  void* vc;
  size_t kv_layer_elems;
  float2* rope;
  float* gpart;
  int ssq_parts_cap;
  size_t gpart_cap;
  unsigned* gcnt;
  size_t gcnt_cap;
  float* apart;
  size_t apart_cap;
  unsigned* acnt;
  size_t acnt_cap;
  // persistent forward pass state (blocks of at most FWD_MAX_M tokens)
  struct Fwd {
    bool on = false;
    unsigned* flags = nullptr;  // all unit flags (zeroed at creation)
    size_t n_flags = 0;
    unsigned *f_qkv, *f_att, *f_o, *f_gu, *f_dn;
    int att_cap = 0;            // attention flags
    unsigned* abort_flag = nullptr;
    float* part[5];             // split-K partials per projection kind (qkv, o, gate_up, down, lm)
    unsigned* cnt[5];
    unsigned epoch = 0;
    unsigned abort_host = 0;    // copy of *abort_flag taken at the last synchronization
    std::map<std::pair<int, int>, std::pair<std::vector<FwdPhase>, FwdPhase*>> tables;  // (K, lm_mode)
  } fw;
  // classifier-free guidance: sequences b and Bi + b are image b's conditional and
  // unconditional streams; decisions use the guided logits
  bool cfg = false;
  float cfg_w = 0.f;
  int Bi = 0;              // images (B, or B / 2 when guided)
  float* mlog = nullptr;   // guided logits [Bi][Kmax][V_img]
  float* mcarry = nullptr; // guided carry [Bi][V_img]
  // decode image buffers
  int* img = nullptr;    // [B][H*W] working grid (absolute ids)
  int img_cap = 0;
  float* qtab = nullptr; // draft logits table for rule C references [B][H*W][V_img]
  size_t qtab_cap = 0;
  float* hs = nullptr;   // head drafting: the state that scored each image token [B][H*W][d]
  size_t hs_cap = 0;
  float* hsrc = nullptr; // head inputs of one draft step [B][W][d] and their tokens [B][W]
  int* tsrc = nullptr;
  // planted drafts (ssd_plant_image): keep flags, replacement codes and the table out [B][H*W]
  unsigned char* pkeep = nullptr;
  int* prepl = nullptr;
  int* ptab = nullptr;
  int* pactive = nullptr;  // [B] sequences still planting (strict decode)
  size_t plant_cap = 0;
};

namespace {

size_t esize(const Dims& dm) { return dm.bf16 ? 2 : 4; }

// ---------------- persistent forward pass ----------------
// Blocks of up to FWD_MAX_M tokens (two 16-token tiles) run the whole backbone
// in one cooperative launch (kernels_fwd.hip); larger token counts use one
// launch per projection and attention.
constexpr int FWD_MAX_M = 32;
constexpr int FWD_MAX_GRID = 512;
constexpr int FWD_KSLICE = 512;  // input features per GEMM work item
constexpr int FWD_FB = 64;       // output features per GEMM work item
constexpr unsigned FWD_SPIN_LIMIT = 1u << 21;  // polls before a wait gives up (seconds)

// shapes whose projections all split into 512-wide K slices and 64-wide feature blocks
bool fwd_shape_ok(const Dims& dm) {
  return dm.bf16 && (dm.D == 64 || dm.D == 128) && dm.d % FWD_KSLICE == 0 && (dm.Hq * dm.D) % FWD_KSLICE == 0 &&
         dm.dff % FWD_KSLICE == 0 && dm.Vimg % FWD_FB == 0 && dm.d / FWD_FB <= 64;  // rms parts of the kernel
}

// split-K partial floats of one projection kind for up to two token tiles
size_t fwd_part_floats(int N, int Kd) { return (size_t)(Kd / FWD_KSLICE) * (N / FWD_FB) * 4 * (2 * 64 * 4); }

// attention flags a session needs: B * Hkv * query groups of the largest persistent block
int fwd_att_units(const Dims& dm, int B, int Kmax) {
  const int K = std::min(Kmax, FWD_MAX_M / B);
  return B * dm.Hkv * ((K * (dm.Hq / dm.Hkv) + 15) / 16);
}

// Grid of the persistent kernel for each tile count and the XCD mapping of a
// cooperative launch (workgroup w on XCD w % X, checked with the kernel's
// own probe), or grid 0 where the kernel cannot run.  The single-launch pass
// is used when SSD_FORWARD=persistent at model creation; otherwise every pass
// runs as one launch per projection and attention.
void setup_fwd(ssd_model* m) {
  const char* env = std::getenv("SSD_FORWARD");
  if (!env || std::strcmp(env, "persistent") != 0) return;
  // SSD_FWD_SPIN_LIMIT lowers the bound of every dependency wait (tests drive
  // the abandoned-wait path with it: the grid still drains, the host reports
  // SSD_E_DEVICE and poisons the session)
  m->fwd_spin_limit = FWD_SPIN_LIMIT;
  if (const char* sl = std::getenv("SSD_FWD_SPIN_LIMIT")) {
    const long v = std::strtol(sl, nullptr, 10);
    if (v >= 0 && v < (long)FWD_SPIN_LIMIT) m->fwd_spin_limit = (unsigned)v;
  }
  if (!fwd_shape_ok(m->dm)) return;
  for (int mt = 1; mt <= 2; ++mt) {
    int g = std::min(fwd_max_grid(mt, m->dm.D), FWD_MAX_GRID);
    g -= g % 8;
    if (g < 64) continue;
    int* d = nullptr;
    if (hipMalloc(&d, (size_t)g * sizeof(int)) != hipSuccess) {
      (void)hipGetLastError();
      continue;
    }
    FwdArgs a{};
    a.n_phases = 0;
    a.probe = d;
    std::vector<int> h(g, -1);
    bool ok = fwd_persistent(a, mt, m->dm.D, g, m->stream) == hipSuccess &&
              hipMemcpyAsync(h.data(), d, (size_t)g * sizeof(int), hipMemcpyDeviceToHost, m->stream) == hipSuccess &&
              hipStreamSynchronize(m->stream) == hipSuccess;
    (void)hipFree(d);
    if (!ok) {
      (void)hipGetLastError();
      continue;
    }
    bool mapped = m->xcd > 0;
    for (int w = 0; w < g && mapped; ++w) mapped = h[w] == w % m->xcd;
    m->fwd_grid[mt - 1] = g;
    m->fwd_xcd[mt - 1] = mapped ? m->xcd : 0;
  }
}

// The abort flag is read where the host synchronizes anyway: fetch enqueues
// the copy, check (after the stream has drained) turns a set flag into an error.
void fwd_abort_fetch(ssd_session* s) {
  if (s->fw.on)
    HIPCHK(hipMemcpyAsync(&s->fw.abort_host, s->fw.abort_flag, sizeof(unsigned), hipMemcpyDeviceToHost, s->stream));
}
void fwd_abort_check(ssd_session* s) {
  if (s->fw.on && s->fw.abort_host)
    throw HipError{hipErrorLaunchTimeOut, "persistent forward pass abandoned a dependency wait"};
}

// A projection as persistent work items: 64 features x (bursts x 512) inputs
// each, with the fewest bursts that keep the items within one round of the
// grid (a burst beyond the first costs its weight load's latency, a second
// round a whole item).
FwdGemm fwd_gemm(const void* W, int N, int Kd, const void* in, size_t in_plane, int ld_in, int M, int X, int grid,
                 float* part, unsigned* cnt, unsigned* out_flags, int out_layer, const EpiArgs& e) {
  FwdGemm g{};
  g.W = W;
  g.N = N;
  g.K = Kd;
  g.KB = Kd / 32;
  g.n_fb = N / FWD_FB;
  const int slices = Kd / FWD_KSLICE;
  g.bursts = 1;
  for (int b = 2; b <= 4; b *= 2)
    if (xcd_grid(g.n_fb, slices / g.bursts, X) > grid && slices % b == 0) g.bursts = b;
  g.S = slices / g.bursts;
  g.items = xcd_grid(g.n_fb, g.S, X);
  g.M = M;
  g.in = (const uint16_t*)in;
  g.in_plane = in_plane;
  g.ld_in = ld_in;
  g.dep_width = FWD_FB;
  g.dep_scale = 1;
  g.part = part;
  g.counters = cnt;
  g.out_flags = out_flags;
  g.out_layer = out_layer;
  g.epi = e;
  return g;
}

// Phase table of one (K, lm_mode): per layer QKV, attention, O, gate/up, down;
// then the output layer.  Flag values are layer + 1 (plus the pass's epoch base).
const FwdPhase* fwd_table(ssd_session* s, int K, int lm_mode, int X, int G, const EpiArgs& base, int att_groups) {
  auto key = std::make_pair(K, lm_mode);
  auto it = s->fw.tables.find(key);
  if (it != s->fw.tables.end()) return it->second.second;
  const Dims& dm = s->dm;
  ssd_model* m = s->m;
  const int B = s->B, M = B * K, d = dm.d, D = dm.D;
  const int Nqkv = (dm.Hq + 2 * dm.Hkv) * D;
  const int nfb_d = d / FWD_FB;
  const size_t es = esize(dm);
  std::vector<FwdPhase> ph;
  for (int l = 0; l < dm.L; ++l) {
    const LayerW& W = m->layers[l];
    char* kc = (char*)s->kc + (size_t)l * s->kv_layer_elems * es;
    char* vc = (char*)s->vc + (size_t)l * s->kv_layer_elems * es;
    FwdPhase p{};
    // QKV projection (+ rotary, KV write): input xn of the previous layer's down projection
    EpiArgs e = base;
    e.kind = EPI_QKV;
    e.ssq = s->ssq;
    e.ssq_parts = l == 0 ? 1 : nfb_d;
    e.q = s->q;
    e.kc = kc;
    e.vc = vc;
    p.kind = FWD_GEMM;
    p.g = fwd_gemm(W.wqkv, Nqkv, d, s->xn, s->xn_plane, d, M, X, G, s->fw.part[0], s->fw.cnt[0], s->fw.f_qkv, l + 1, e);
    if (l > 0) {
      p.g.dep = s->fw.f_dn;
      p.g.dep_layer = l;
      p.g.rms_dep = s->fw.f_dn;
      p.g.rms_units = nfb_d;
      p.g.rms_layer = l;
    }
    ph.push_back(p);
    // attention over the cache of layer l
    p = FwdPhase{};
    p.kind = FWD_ATTN;
    p.a.dep = s->fw.f_qkv;
    p.a.dep_width = FWD_FB;
    p.a.qN = dm.Hq * D;
    p.a.kN = dm.Hkv * D;
    p.a.layer = l + 1;
    p.a.kc = kc;
    p.a.vc = vc;
    p.a.out_flags = s->fw.f_att;
    ph.push_back(p);
    // O projection + residual: needs every attention output
    e = base;
    e.kind = EPI_RESID;
    e.ssq = nullptr;
    e.gnext = W.g2;
    e.ld = d;
    p = FwdPhase{};
    p.kind = FWD_GEMM;
    p.g = fwd_gemm(W.wo, d, dm.Hq * D, s->o, s->o_plane, dm.Hq * D, M, X, G, s->fw.part[1], s->fw.cnt[1], s->fw.f_o, l + 1,
                   e);
    p.g.dep = s->fw.f_att;
    p.g.dep_att = 1;
    p.g.dep_layer = l + 1;
    ph.push_back(p);
    // gate/up + SwiGLU
    e = base;
    e.kind = EPI_SWIGLU;
    e.ssq = s->ssq;
    e.ssq_parts = nfb_d;
    e.h = s->h;
    e.ld = dm.dff;
    p = FwdPhase{};
    p.kind = FWD_GEMM;
    p.g = fwd_gemm(W.w13, 2 * dm.dff, d, s->xn, s->xn_plane, d, M, X, G, s->fw.part[2], s->fw.cnt[2], s->fw.f_gu, l + 1,
                   e);
    p.g.dep = s->fw.f_o;
    p.g.dep_layer = l + 1;
    p.g.rms_dep = s->fw.f_o;
    p.g.rms_units = nfb_d;
    p.g.rms_layer = l + 1;
    ph.push_back(p);
    // down projection + residual: h feature j comes from gate/up block j / 32
    e = base;
    e.kind = EPI_RESID;
    e.ssq = nullptr;
    e.gnext = (l + 1 < dm.L) ? m->layers[l + 1].g1 : m->gf;
    e.ld = d;
    p = FwdPhase{};
    p.kind = FWD_GEMM;
    p.g = fwd_gemm(W.w2, d, dm.dff, s->h, s->h_plane, dm.dff, M, X, G, s->fw.part[3], s->fw.cnt[3], s->fw.f_dn, l + 1, e);
    p.g.dep = s->fw.f_gu;
    p.g.dep_scale = 2;
    p.g.dep_layer = l + 1;
    ph.push_back(p);
  }
  // output layer over all rows (lm_mode 0) or the last row of each sequence
  EpiArgs e = base;
  e.kind = EPI_LOGITS;
  e.ssq = s->ssq;
  e.ssq_parts = nfb_d;
  e.logits = s->logits;
  e.ld = dm.Vimg;
  FwdPhase p{};
  p.kind = FWD_GEMM;
  if (lm_mode == 0) {
    p.g = fwd_gemm(m->wlm, dm.Vimg, d, s->xn, s->xn_plane, d, M, X, G, s->fw.part[4], s->fw.cnt[4], nullptr, 0, e);
  } else {
    e.ssq_off = K - 1;
    e.ssq_step = K;
    p.g = fwd_gemm(m->wlm, dm.Vimg, d, (const uint16_t*)s->xn + (size_t)(K - 1) * d, s->xn_plane, K * d, B, X, G,
                   s->fw.part[4], s->fw.cnt[4], nullptr, 0, e);
  }
  p.g.dep = s->fw.f_dn;
  p.g.dep_layer = dm.L;
  p.g.rms_dep = s->fw.f_dn;
  p.g.rms_units = nfb_d;
  p.g.rms_layer = dm.L;
  ph.push_back(p);
  // rotations: each phase starts on the workgroups after the previous phase's
  // items (attention counts its query groups, its fewest items)
  int R = 0;
  for (FwdPhase& q : ph) {
    q.rot = R;
    const int n = q.kind == FWD_GEMM ? q.g.items : ((att_groups + 7) / 8) * 8;
    R = (R + n) % G;
  }
  FwdPhase* dev = s->mem.get<FwdPhase>(ph.size());
  auto& slot = s->fw.tables[key];
  slot.first = std::move(ph);
  slot.second = dev;
  HIPCHK(hipMemcpyAsync(dev, slot.first.data(), slot.first.size() * sizeof(FwdPhase), hipMemcpyHostToDevice,
                        s->stream));
  return dev;
}

// ---------------- forward pass ----------------
// lm_mode: 0 = logits for all B*K rows; 1 = logits for the last row of each sequence only
void run_forward(ssd_session* s, int K, int lm_mode) {
  const Dims& dm = s->dm;
  ssd_model* m = s->m;
  hipStream_t st = s->stream;
  const int B = s->B, M = B * K;
  const int d = dm.d, D = dm.D;
  const int Nqkv = (dm.Hq + 2 * dm.Hkv) * D;
  const size_t es = esize(dm);
  int max_ctx_now = 0;
  for (int b = 0; b < B; ++b) max_ctx_now = std::max(max_ctx_now, s->f[b] + K);

  embed(dm, m->emb, s->tok, M, m->layers[0].g1, s->x, s->xn, s->xn_plane, s->ssq, st);
  int ssq_parts = 1;

  EpiArgs base{};
  base.Kblk = K;
  base.f = s->d_f;
  base.ssq_ld = s->ssq_rows_ld;
  base.ssq_off = 0;
  base.ssq_step = 1;
  base.inv_d = 1.0f / (float)d;
  base.eps = dm.eps;
  base.Lmax = s->Lmax;
  base.Hq = dm.Hq;
  base.Hkv = dm.Hkv;
  base.D = D;
  base.qrows_pad = q_rows_pad(K, dm.Hq / dm.Hkv);
  base.rope = s->rope;
  base.x = s->x;
  base.xn = s->xn;
  base.ssq_out = s->ssq;
  base.ssq_out_ld = s->ssq_rows_ld;
  base.q_plane = s->q_plane;
  base.xn_plane = s->xn_plane;
  base.h_plane = s->h_plane;

  if (dm.bf16) {
    // algorithmic bytes: bf16 weights and KV, 4-byte activations (two bf16 planes), fp32 residual
    const double A = 4.0;
    const int X = m->xcd;
    GemmPlan pq = gemm_plan_bf16(M, Nqkv, d, X);
    GemmPlan po = gemm_plan_bf16(M, d, dm.Hq * D, X);
    GemmPlan p13 = gemm_plan_bf16(M, 2 * dm.dff, d, X);
    GemmPlan p2 = gemm_plan_bf16(M, d, dm.dff, X);
    AttnPlan pa = attn_plan(dm, B, K, max_ctx_now, X);
    // workspaces were sized at session creation for every plan the session can
    // meet; a plan outside them is a bug, refused before any launch
    auto need = [](bool ok, const char* what) {
      if (!ok) throw HipError{hipErrorInvalidValue, what};
    };
    need(M <= s->Mmax, "token count exceeds the session's activation buffers");
    for (const GemmPlan* gp : {&pq, &po, &p13, &p2}) {
      need(gemm_partials_floats(*gp, M) <= s->gpart_cap && (size_t)gemm_counters(*gp) <= s->gcnt_cap,
           "GEMM plan exceeds the split-K workspace");
    }
    need(po.n_fb <= s->ssq_parts_cap && p2.n_fb <= s->ssq_parts_cap, "rms partial sums exceed their buffer");
    need(attn_partials_floats(dm, pa, B) <= s->apart_cap && (size_t)B * dm.Hkv * pa.nqg <= s->acnt_cap,
         "attention plan exceeds its workspace");
    double attn_bytes = 2.0 * M * dm.Hq * D * A;  // q read + o written
    double attn_flops = 0.0;                       // QK^T and PV over the visible keys
    for (int b = 0; b < B; ++b) {
      attn_bytes += 2.0 * (s->f[b] + K) * dm.Hkv * D * es;
      attn_flops += 4.0 * dm.Hq * D * ((double)s->f[b] * K + 0.5 * K * (K + 1));
    }
    const double qkv_bytes = (double)Nqkv * d * es + (double)M * d * A + (double)M * dm.Hq * D * A +
                             2.0 * M * dm.Hkv * D * es;
    const double o_bytes = (double)d * dm.Hq * D * es + (double)M * dm.Hq * D * A + (double)M * d * (8 + A);
    const double gu_bytes = 2.0 * dm.dff * d * es + (double)M * d * A + (double)M * dm.dff * A;
    const double dn_bytes = (double)d * dm.dff * es + (double)M * dm.dff * A + (double)M * d * (8 + A);
    const int mt = M <= 16 ? 1 : 2;
    if (s->fw.on && M <= FWD_MAX_M && m->fwd_grid[mt - 1] > 0) {
      const int G = m->fwd_grid[mt - 1], XF = m->fwd_xcd[mt - 1];
      AttnPlan pf = attn_plan(dm, B, K, max_ctx_now, XF, G);
      const int groups = B * dm.Hkv * pf.nqg;
      need(attn_partials_floats(dm, pf, B) <= s->apart_cap && (size_t)groups <= s->acnt_cap && groups <= s->fw.att_cap,
           "attention plan exceeds its workspace");
      need(d / FWD_FB <= s->ssq_parts_cap, "rms partial sums exceed their buffer");
      const FwdPhase* tab = fwd_table(s, K, lm_mode, XF, G, base, groups);
      FwdArgs a{};
      a.phases = tab;
      a.n_phases = 5 * dm.L + 1;
      a.xcd = XF;
      a.abort_flag = s->fw.abort_flag;
      a.spin_limit = m->fwd_spin_limit;
      // flag values of this pass lie above every value an earlier pass stored;
      // before they would wrap, the flags restart from zero
      if ((uint64_t)(s->fw.epoch + 2) * (dm.L + 1) >= (1ull << 32)) {
        fill_u32(s->fw.flags, s->fw.n_flags, 0u, st);
        s->fw.epoch = 0;
      }
      ++s->fw.epoch;
      a.epoch_base = s->fw.epoch * (unsigned)(dm.L + 1);
      a.att = attn_args(dm, pf, B, K, s->d_f, s->q, s->q_plane, nullptr, nullptr, s->Lmax, s->o, s->o_plane, s->apart,
                        s->acnt);
      a.att_items = attn_items(a.att);
      const int rows_lm = lm_mode == 0 ? M : B;
      const double lm_bytes = (double)dm.Vimg * d * es + (double)rows_lm * d * A + (double)rows_lm * dm.Vimg * 4;
      const double fwd_bytes = dm.L * (qkv_bytes + attn_bytes + o_bytes + gu_bytes + dn_bytes) + lm_bytes;
      m->prof.run(6, fwd_bytes, st, [&] { HIPCHK(fwd_persistent(a, mt, D, G, st)); });
      HIPCHK(hipGetLastError());
      return;
    }
    for (int l = 0; l < dm.L; ++l) {
      const LayerW& W = m->layers[l];
      char* kc = (char*)s->kc + (size_t)l * s->kv_layer_elems * es;
      char* vc = (char*)s->vc + (size_t)l * s->kv_layer_elems * es;
      EpiArgs e = base;
      e.kind = EPI_QKV;
      e.ssq = s->ssq;
      e.ssq_parts = ssq_parts;
      e.q = s->q;
      e.kc = kc;
      e.vc = vc;
      m->prof.run(0, qkv_bytes, st, [&] {
        gemm_bf16(pq, W.wqkv, Nqkv, d, s->xn, s->xn_plane, d, M, e, s->gpart, s->gcnt, st);
      }, 2.0 * M * Nqkv * d, pq.tile);
      m->prof.run(5, attn_bytes, st, [&] {
        attention_bf16(dm, pa, B, K, s->d_f, s->q, s->q_plane, kc, vc, s->Lmax, s->o, s->o_plane, s->apart, s->acnt,
                       st);
      }, attn_flops);
      e = base;
      e.kind = EPI_RESID;
      e.ssq = nullptr;
      e.gnext = W.g2;
      e.ld = d;
      m->prof.run(1, o_bytes, st, [&] {
        gemm_bf16(po, W.wo, d, dm.Hq * D, s->o, s->o_plane, dm.Hq * D, M, e, s->gpart, s->gcnt, st);
      }, 2.0 * M * d * dm.Hq * D, po.tile);
      ssq_parts = po.n_fb;
      e = base;
      e.kind = EPI_SWIGLU;
      e.ssq = s->ssq;
      e.ssq_parts = ssq_parts;
      e.h = s->h;
      e.ld = dm.dff;
      m->prof.run(2, gu_bytes, st, [&] {
        gemm_bf16(p13, W.w13, 2 * dm.dff, d, s->xn, s->xn_plane, d, M, e, s->gpart, s->gcnt, st);
      }, 2.0 * M * 2 * dm.dff * d, p13.tile);
      e = base;
      e.kind = EPI_RESID;
      e.ssq = nullptr;
      e.gnext = (l + 1 < dm.L) ? m->layers[l + 1].g1 : m->gf;
      e.ld = d;
      m->prof.run(3, dn_bytes, st, [&] {
        gemm_bf16(p2, W.w2, d, dm.dff, s->h, s->h_plane, dm.dff, M, e, s->gpart, s->gcnt, st);
      }, 2.0 * M * d * dm.dff, p2.tile);
      ssq_parts = p2.n_fb;
    }
    EpiArgs e = base;
    e.kind = EPI_LOGITS;
    e.ssq = s->ssq;
    e.ssq_parts = ssq_parts;
    e.logits = s->logits;
    e.ld = dm.Vimg;
    if (lm_mode == 0) {
      GemmPlan pl = gemm_plan_bf16(M, dm.Vimg, d, X);
      if (gemm_partials_floats(pl, M) > s->gpart_cap || (size_t)gemm_counters(pl) > s->gcnt_cap)
        throw HipError{hipErrorInvalidValue, "GEMM plan exceeds the split-K workspace"};
      m->prof.run(4, (double)dm.Vimg * d * es + (double)M * d * A + (double)M * dm.Vimg * 4, st, [&] {
        gemm_bf16(pl, m->wlm, dm.Vimg, d, s->xn, s->xn_plane, d, M, e, s->gpart, s->gcnt, st);
      }, 2.0 * M * dm.Vimg * d, pl.tile);
    } else {
      e.ssq_off = K - 1;
      e.ssq_step = K;
      GemmPlan pl = gemm_plan_bf16(B, dm.Vimg, d, X);
      if (gemm_partials_floats(pl, B) > s->gpart_cap || (size_t)gemm_counters(pl) > s->gcnt_cap)
        throw HipError{hipErrorInvalidValue, "GEMM plan exceeds the split-K workspace"};
      m->prof.run(4, (double)dm.Vimg * d * es + (double)B * d * A + (double)B * dm.Vimg * 4, st, [&] {
        gemm_bf16(pl, m->wlm, dm.Vimg, d, (const uint16_t*)s->xn + (size_t)(K - 1) * d, s->xn_plane, K * d, B, e,
                  s->gpart, s->gcnt, st);
      }, 2.0 * B * dm.Vimg * d, pl.tile);
    }
  } else {
    for (int l = 0; l < dm.L; ++l) {
      const LayerW& W = m->layers[l];
      float* kc = (float*)s->kc + (size_t)l * s->kv_layer_elems;
      float* vc = (float*)s->vc + (size_t)l * s->kv_layer_elems;
      EpiArgs e = base;
      e.kind = EPI_QKV;
      e.ssq = s->ssq;
      e.ssq_parts = 1;
      e.q = s->q;
      e.kc = kc;
      e.vc = vc;
      gemm_f32((const float*)W.wqkv, Nqkv, d, (const float*)s->xn, d, M, e, st);
      attention_f32(dm, B, K, s->d_f, (const float*)s->q, kc, vc, s->Lmax, (float*)s->o, st);
      e = base;
      e.kind = EPI_RESID;
      e.ssq = nullptr;
      e.gnext = W.g2;
      e.ld = d;
      gemm_f32((const float*)W.wo, d, dm.Hq * D, (const float*)s->o, dm.Hq * D, M, e, st);
      norm_rows_f32(s->x, M, d, nullptr, nullptr, s->ssq, st);
      e = base;
      e.kind = EPI_SWIGLU;
      e.ssq = s->ssq;
      e.ssq_parts = 1;
      e.h = s->h;
      e.ld = dm.dff;
      gemm_f32((const float*)W.w13, 2 * dm.dff, d, (const float*)s->xn, d, M, e, st);
      e = base;
      e.kind = EPI_RESID;
      e.ssq = nullptr;
      e.gnext = (l + 1 < dm.L) ? m->layers[l + 1].g1 : m->gf;
      e.ld = d;
      gemm_f32((const float*)W.w2, d, dm.dff, (const float*)s->h, dm.dff, M, e, st);
      norm_rows_f32(s->x, M, d, nullptr, nullptr, s->ssq, st);
    }
    EpiArgs e = base;
    e.kind = EPI_LOGITS;
    e.ssq = s->ssq;
    e.ssq_parts = 1;
    e.logits = s->logits;
    e.ld = dm.Vimg;
    if (lm_mode == 0) {
      gemm_f32((const float*)m->wlm, dm.Vimg, d, (const float*)s->xn, d, M, e, st);
    } else {
      e.ssq_off = K - 1;
      e.ssq_step = K;
      gemm_f32((const float*)m->wlm, dm.Vimg, d, (const float*)s->xn + (size_t)(K - 1) * d, K * d, B, e, st);
    }
  }
  HIPCHK(hipGetLastError());
}

// Number of XCDs if workgroup w always runs on XCD w % X (checked on 4096
// workgroups through the XCC_ID register), else 0 -- the cross-workgroup
// reductions then fall back to device-scope fences.  SSD_NO_XCD_LOCAL=1 forces
// the fallback.
int detect_xcd(hipStream_t st) {
  const char* env = std::getenv("SSD_NO_XCD_LOCAL");
  if (env && env[0] == '1') return 0;
  const int n = 4096;
  int* d = nullptr;
  if (hipMalloc(&d, n * sizeof(int)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  xcc_probe(d, n, st);
  std::vector<int> h(n, -1);
  bool ok = hipGetLastError() == hipSuccess &&
            hipMemcpyAsync(h.data(), d, n * sizeof(int), hipMemcpyDeviceToHost, st) == hipSuccess &&
            hipStreamSynchronize(st) == hipSuccess;
  (void)hipFree(d);
  if (!ok) {
    (void)hipGetLastError();
    return 0;
  }
  int X = 0;
  for (int v : h) X = std::max(X, v + 1);
  if (X < 1) return 0;
  for (int w = 0; w < n; ++w)
    if (h[w] != w % X) return 0;
  return X;
}

// workspace sizes for a session that runs blocks of up to Kmax tokens and a prefill of P
void size_workspaces(const Dims& dm, const ssd_model* m, int B, int P, int Kmax, int Lmax, size_t& gpart, size_t& gcnt,
                     size_t& apart, size_t& acnt, int& ssq_parts_max) {
  gpart = 0;
  gcnt = 0;
  apart = 0;
  acnt = 0;
  ssq_parts_max = 1;
  if (!dm.bf16) return;
  const int Nqkv = (dm.Hq + 2 * dm.Hkv) * dm.D;
  // every token-tile class a plan can fall in: up to 16, 32 and 64 tokens,
  // 65..128 (64-token tiles), beyond 128 (tiled, every row-tile count up to
  // where no plan splits K any more)
  for (int Mc : gemm_row_classes()) {
    for (auto nk : {std::make_pair(Nqkv, dm.d), std::make_pair(dm.d, dm.Hq * dm.D), std::make_pair(2 * dm.dff, dm.d),
                    std::make_pair(dm.d, dm.dff), std::make_pair(dm.Vimg, dm.d)}) {
      GemmPlan p = gemm_plan_bf16(Mc, nk.first, nk.second, 0);  // sizes do not depend on the XCD mapping
      gpart = std::max(gpart, gemm_partials_floats(p, Mc));
      gcnt = std::max(gcnt, (size_t)gemm_counters(p));
      if (nk.first == dm.d) ssq_parts_max = std::max(ssq_parts_max, std::max(p.n_fb, gemm_max_parts(dm.d)));
    }
  }
  // every block length the session can run, every context up to Lmax
  std::vector<int> Ks;
  for (int K = 1; K <= Kmax; ++K) Ks.push_back(K);
  Ks.push_back(P);
  for (int K : Ks) {
    for (int ctx = 1; ctx <= Lmax; ++ctx) {
      AttnPlan pc = attn_plan(dm, B, K, ctx, 0);
      apart = std::max(apart, attn_partials_floats(dm, pc, B));
      acnt = std::max(acnt, (size_t)B * dm.Hkv * pc.nqg);
    }
    AttnPlan pa = attn_plan(dm, B, K, Lmax, 0);
    apart = std::max(apart, attn_partials_floats(dm, pa, B));
    acnt = std::max(acnt, (size_t)B * dm.Hkv * pa.nqg);
  }
  // the persistent forward pass: its own attention plans and one rms part per 64 features
  for (int mt = 1; mt <= 2; ++mt) {
    const int G = m->fwd_grid[mt - 1];
    if (G == 0) continue;
    ssq_parts_max = std::max(ssq_parts_max, dm.d / FWD_FB);
    for (int K : Ks) {
      if ((long)B * K > 16 * mt || (long)B * K <= 16 * (mt - 1)) continue;
      for (int X : {0, m->fwd_xcd[mt - 1]}) {
        for (int ctx = 1; ctx <= Lmax; ++ctx) {
          AttnPlan pc = attn_plan(dm, B, K, ctx, X, G);
          apart = std::max(apart, attn_partials_floats(dm, pc, B));
          acnt = std::max(acnt, (size_t)B * dm.Hkv * pc.nqg);
        }
      }
    }
  }
}

ssd_status create_session(ssd_model* m, int B, int P, int Lmax_req, int Kmax, hipStream_t stream, ssd_session** out) {
  const Dims& dm = m->dm;
  auto* s = new ssd_session();
  s->m = m;
  s->dm = dm;
  s->stream = stream;
  s->B = B;
  s->Bi = B;
  s->P = P;
  s->Lmax = ((Lmax_req + 63) / 64) * 64;
  s->max_ctx = Lmax_req;
  s->Kmax = Kmax;
  s->Mmax = B * std::max(P, Kmax);
  s->ring = Kmax;
  s->f.assign(B, 0);
  const size_t es = esize(dm);
  try {
    size_t gpart, gcnt, apart, acnt;
    int ssq_parts;
    size_workspaces(dm, m, B, P, Kmax, s->Lmax, gpart, gcnt, apart, acnt, ssq_parts);
    const size_t M = s->Mmax;
    s->d_f = s->mem.get<int>(B);
    s->tok = s->mem.get<int>(M);
    s->acc = s->mem.get<unsigned char>(M);
    s->cnt = s->mem.get<int>((size_t)NCNT_ROUNDS * B);  // [round of the block][B] in image decodes
    s->amax = s->mem.get<int>(M);
    s->x = s->mem.get<float>(M * dm.d);
    // activations: 4 bytes per element (fp32, or hi + lo bf16 planes)
    s->xn_plane = M * dm.d;
    // q: the tiled bf16 layout pads each KV head's K*g query rows to 32; fp32 uses M*Hq*D of it
    const size_t qcap = (size_t)B * dm.Hkv * q_rows_pad(std::max(P, Kmax), dm.Hq / dm.Hkv) * dm.D;
    s->q_plane = qcap;
    s->o_plane = M * dm.Hq * dm.D;
    s->h_plane = M * dm.dff;
    s->xn = s->mem.get<char>(M * dm.d * 4);
    s->ssq_rows_ld = (int)M;
    s->ssq = s->mem.get<float>((size_t)ssq_parts * M);
    s->ssq_parts_cap = ssq_parts;
    s->q = s->mem.get<char>(qcap * 4);
    s->o = s->mem.get<char>(M * dm.Hq * dm.D * 4);
    s->h = s->mem.get<char>(M * dm.dff * 4);
    s->logits = s->mem.get<float>(M * dm.Vimg);
    s->carry = s->mem.get<float>((size_t)B * dm.Vimg);
    s->ref = s->mem.get<float>((size_t)B * s->ring * dm.Vimg);
    s->refstage = s->mem.get<float>((size_t)B * Kmax * dm.Vimg);
    s->ref_flag = s->mem.get<int>((size_t)B * s->ring);
    s->kv_layer_elems = (size_t)B * dm.Hkv * s->Lmax * dm.D;
    s->kc = s->mem.get<char>(s->kv_layer_elems * dm.L * es);
    s->vc = s->mem.get<char>(s->kv_layer_elems * dm.L * es);
    s->rope = s->mem.get<float2>((size_t)s->Lmax * (dm.D / 2));
    s->gpart_cap = gpart;
    s->gpart = s->mem.get<float>(gpart);
    s->gcnt_cap = gcnt;
    s->gcnt = s->mem.get<unsigned>(gcnt);
    s->apart_cap = apart;
    s->apart = s->mem.get<float>(apart);
    s->acnt_cap = acnt;
    s->acnt = s->mem.get<unsigned>(acnt);
    hipStream_t st = s->stream;
    // the persistent kernel addresses activations and caches through buffer
    // resources: every array must stay below 2 GiB
    const size_t lim = (size_t)1 << 31;
    const bool fits = s->kv_layer_elems * es < lim && M * dm.d * 4 < lim && qcap * 4 < lim &&
                      M * dm.Hq * dm.D * 4 < lim && M * dm.dff * 4 < lim && M * dm.Vimg * 4 < lim &&
                      (size_t)ssq_parts * M * 4 < lim;
    if (dm.bf16 && (m->fwd_grid[0] > 0 || m->fwd_grid[1] > 0) && B <= FWD_MAX_M && fits) {
      auto& fw = s->fw;
      const int Nqkv = (dm.Hq + 2 * dm.Hkv) * dm.D;
      const int nq = Nqkv / FWD_FB, nd = dm.d / FWD_FB, ng = 2 * dm.dff / FWD_FB;
      fw.att_cap = fwd_att_units(dm, B, Kmax);
      const int n_cnt[5] = {nq, nd, ng, nd, dm.Vimg / FWD_FB};
      fw.n_flags = (size_t)nq + fw.att_cap + nd + ng + nd + 1;
      for (int c : n_cnt) fw.n_flags += c;
      fw.flags = s->mem.get<unsigned>(fw.n_flags);
      unsigned* f = fw.flags;
      fw.f_qkv = f;
      f += nq;
      fw.f_att = f;
      f += fw.att_cap;
      fw.f_o = f;
      f += nd;
      fw.f_gu = f;
      f += ng;
      fw.f_dn = f;
      f += nd;
      fw.abort_flag = f;
      f += 1;
      // split counters live in the same zeroed block (they re-arm themselves)
      for (int k = 0; k < 5; ++k) {
        fw.cnt[k] = f;
        f += n_cnt[k];
      }
      const int NK[5][2] = {{Nqkv, dm.d}, {dm.d, dm.Hq * dm.D}, {2 * dm.dff, dm.d}, {dm.d, dm.dff}, {dm.Vimg, dm.d}};
      for (int k = 0; k < 5; ++k) fw.part[k] = s->mem.get<float>(fwd_part_floats(NK[k][0], NK[k][1]));
      fill_u32(fw.flags, fw.n_flags, 0u, st);
      fw.on = true;
    }
    // zero state that kernels read before writing (KV slots beyond the context are multiplied by 0)
    fill_u32((unsigned*)s->kc, s->kv_layer_elems * dm.L * es / 4, 0u, st);
    fill_u32((unsigned*)s->vc, s->kv_layer_elems * dm.L * es / 4, 0u, st);
    fill_u32((unsigned*)s->ref_flag, (size_t)B * s->ring, 0u, st);
    fill_u32((unsigned*)s->q, qcap, 0u, st);  // padded query rows are read (and masked) by attention
    fill_u32(s->gcnt, gcnt, 0u, st);
    fill_u32(s->acnt, acnt, 0u, st);
    fill_u32((unsigned*)s->d_f, B, 0u, st);
    // rotary table (host double precision, rounded to fp32)
    std::vector<float2> rope((size_t)s->Lmax * (dm.D / 2));
    for (int p = 0; p < s->Lmax; ++p)
      for (int j = 0; j < dm.D / 2; ++j) {
        double inv = std::pow((double)dm.theta, -2.0 * j / dm.D);
        double ang = (double)p * inv;
        rope[(size_t)p * (dm.D / 2) + j] = make_float2((float)std::cos(ang), (float)std::sin(ang));
      }
    HIPCHK(hipMemcpyAsync(s->rope, rope.data(), rope.size() * sizeof(float2), hipMemcpyHostToDevice, st));
    HIPCHK(hipStreamSynchronize(st));
    HIPCHK(hipGetLastError());
  } catch (HipError& e) {
    delete s;
    if (e.e == hipErrorOutOfMemory || std::string(e.what) == "hipMalloc")
      return fail(SSD_E_OOM, "device allocation failed (%s)", hipGetErrorString(e.e));
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  *out = s;
  return SSD_OK;
}

// prefix pass: tokens already in s->tok as [B][P]
void prefill_pass(ssd_session* s) {
  run_forward(s, s->P, 1);
  commit_update(s->B, -s->P, s->dm.Vimg, s->logits, s->carry, s->d_f, s->ref_flag, s->ring, s->stream);
  for (int b = 0; b < s->B; ++b) s->f[b] = s->P;
}

ssd_status check_tokens_host(const int32_t* t, size_t n, int lo, int hi, const char* what) {
  for (size_t i = 0; i < n; ++i)
    if (t[i] < lo || t[i] >= hi) return fail(SSD_E_INVAL, "%s[%zu] = %d outside [%d, %d)", what, i, t[i], lo, hi);
  return SSD_OK;
}

}  // namespace

extern "C" {

const char* ssd_last_error(void) { return g_err.c_str(); }

int64_t ssd_weights_numel(const ssd_model_config* cfg) {
  if (validate_config(cfg) != SSD_OK) return -1;
  return numel_of(*cfg);
}

ssd_status ssd_init_model(const ssd_model_config* cfg, const void* weights, void* stream, ssd_model** out) {
  g_err.clear();
  if (!out) return fail(SSD_E_INVAL, "out is NULL");
  *out = nullptr;
  ssd_status vs = validate_config(cfg);
  if (vs != SSD_OK) return vs;
  if (!weights) return fail(SSD_E_INVAL, "weights is NULL");
  auto* m = new ssd_model();
  m->cfg = *cfg;
  Dims& dm = m->dm;
  dm.L = cfg->n_layers;
  dm.d = cfg->d_model;
  dm.Hq = cfg->n_heads;
  dm.Hkv = cfg->n_kv_heads;
  dm.D = cfg->head_dim;
  dm.dff = cfg->d_ff;
  dm.V = cfg->vocab;
  dm.img_lo = cfg->img_lo;
  dm.img_hi = cfg->img_hi;
  dm.Vimg = cfg->img_hi - cfg->img_lo;
  dm.bf16 = cfg->dtype == SSD_BF16;
  dm.eps = cfg->rms_eps;
  dm.theta = cfg->rope_theta;
  m->stream = (hipStream_t)stream;
  const size_t es = esize(dm);
  const int d = dm.d, D = dm.D, f = dm.dff;
  const int Nqkv = (dm.Hq + 2 * dm.Hkv) * D;
  try {
    hipStream_t st = m->stream;
    // offsets (elements) of the packed layout
    const size_t n_emb = (size_t)dm.V * d;
    const size_t n_layer = d + (size_t)Nqkv * d + (size_t)d * dm.Hq * D + d + 2 * (size_t)f * d + (size_t)d * f;
    size_t max_seg = std::max({(size_t)Nqkv * d, (size_t)d * dm.Hq * D, 2 * (size_t)f * d, (size_t)d * f,
                               (size_t)dm.Vimg * d});
    Allocs tmp;
    char* stage = tmp.get<char>(max_seg * es);
    float* gtmp = tmp.get<float>(d);
    // row maps
    std::vector<int> map_qkv(Nqkv), map_13(2 * f), map_id(std::max({d, dm.Vimg, 2 * f, Nqkv}));
    for (int n = 0; n < Nqkv; ++n) {
      if (n < (dm.Hq + dm.Hkv) * D) {
        int head = n / D, r = n % D;
        map_qkv[n] = head * D + ((r % 2 == 0) ? r / 2 : D / 2 + r / 2);
      } else {
        map_qkv[n] = n;
      }
    }
    for (int n = 0; n < 2 * f; ++n) map_13[n] = (n % 2 == 0) ? n / 2 : f + n / 2;
    for (size_t n = 0; n < map_id.size(); ++n) map_id[n] = (int)n;
    int* d_map_qkv = tmp.get<int>(Nqkv);
    int* d_map_13 = tmp.get<int>(2 * f);
    int* d_map_id = tmp.get<int>(map_id.size());
    HIPCHK(hipMemcpy(d_map_qkv, map_qkv.data(), Nqkv * sizeof(int), hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(d_map_13, map_13.data(), 2 * f * sizeof(int), hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(d_map_id, map_id.data(), map_id.size() * sizeof(int), hipMemcpyHostToDevice));

    const char* src = (const char*)weights;
    auto seg = [&](size_t off_elems) { return src + off_elems * es; };
    auto gain = [&](size_t off) -> float* {
      float* g = m->mem.get<float>(d);
      if (dm.bf16) {
        std::vector<uint16_t> hb(d);
        HIPCHK(hipMemcpy(hb.data(), seg(off), d * 2, hipMemcpyDefault));
        std::vector<float> hf(d);
        for (int i = 0; i < d; ++i) {
          uint32_t u = (uint32_t)hb[i] << 16;
          std::memcpy(&hf[i], &u, 4);
        }
        HIPCHK(hipMemcpy(g, hf.data(), d * 4, hipMemcpyHostToDevice));
      } else {
        HIPCHK(hipMemcpy(g, seg(off), d * 4, hipMemcpyDefault));
      }
      return g;
    };
    (void)gtmp;
    // packs the N x K matrix at element offset `off` with `map`
    auto pack = [&](size_t off, int N, int K, const int* dmap) -> void* {
      HIPCHK(hipMemcpy(stage, seg(off), (size_t)N * K * es, hipMemcpyDefault));
      void* dst = m->mem.get<char>((size_t)N * K * es);
      if (dm.bf16)
        pack_bf16_tiles((const uint16_t*)stage, dmap, N, K, dst, st);
      else
        gather_rows_f32((const float*)stage, dmap, N, K, (float*)dst, st);
      HIPCHK(hipGetLastError());
      HIPCHK(hipStreamSynchronize(st));
      return dst;
    };
    m->emb = m->mem.get<char>(n_emb * es);
    HIPCHK(hipMemcpy(m->emb, seg(0), n_emb * es, hipMemcpyDefault));
    size_t off = n_emb;
    m->layers.resize(dm.L);
    for (int l = 0; l < dm.L; ++l) {
      LayerW& W = m->layers[l];
      W.g1 = gain(off);
      off += d;
      W.wqkv = pack(off, Nqkv, d, d_map_qkv);
      off += (size_t)Nqkv * d;
      W.wo = pack(off, d, dm.Hq * D, d_map_id);
      off += (size_t)d * dm.Hq * D;
      W.g2 = gain(off);
      off += d;
      W.w13 = pack(off, 2 * f, d, d_map_13);
      off += 2 * (size_t)f * d;
      W.w2 = pack(off, d, f, d_map_id);
      off += (size_t)d * f;
    }
    (void)n_layer;
    m->gf = gain(off);
    off += d;
    m->wlm = pack(off + (size_t)dm.img_lo * d, dm.Vimg, d, d_map_id);
    if (dm.bf16) {
      m->xcd = detect_xcd(st);
      setup_fwd(m);
    }
    off += (size_t)dm.V * d;
    if ((int64_t)off != numel_of(*cfg)) throw HipError{hipErrorInvalidValue, "layout size mismatch"};
    HIPCHK(hipStreamSynchronize(st));
    m->scratch = scratch_of_current_device();  // set-up of the allocation-free head runs
  } catch (HipError& e) {
    delete m;
    if (e.e == hipErrorOutOfMemory || std::string(e.what) == "hipMalloc")
      return fail(SSD_E_OOM, "device allocation failed (%s)", hipGetErrorString(e.e));
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  *out = m;
  return SSD_OK;
}

void ssd_free_session(ssd_session* s) {
  if (!s) return;
  if (s->m && s->m->dec == s) s->m->dec = nullptr;
  (void)hipStreamSynchronize(s->stream);
  delete s;
}

void ssd_free_model(ssd_model* m) {
  if (!m) return;
  (void)hipStreamSynchronize(m->stream);
  if (m->dec) {
    ssd_session* s = m->dec;
    m->dec = nullptr;
    delete s;
  }
  delete m;
}

ssd_status ssd_prefill(ssd_model* m, int32_t B, int32_t P, const int32_t* prefix, int32_t max_ctx, int32_t max_block,
                       void* stream, ssd_session** out) {
  g_err.clear();
  if (!m || !prefix || !out) return fail(SSD_E_INVAL, "NULL argument");
  *out = nullptr;
  if (m->poisoned) return fail(SSD_E_STATE, "model is poisoned by an earlier device error");
  if (B < 1 || B >= (1 << 20) || P < 1 || max_block < 1) return fail(SSD_E_INVAL, "bad B/P/max_block");
  if (max_ctx < P + 1 || max_ctx >= (1 << 24)) return fail(SSD_E_INVAL, "max_ctx must be in [P+1, 2^24)");
  if (!m->dm.bf16 && max_ctx > 4096) return fail(SSD_E_INVAL, "fp32 models support max_ctx <= 4096");
  std::vector<int32_t> host((size_t)B * P);
  if (hipMemcpy(host.data(), prefix, host.size() * 4, hipMemcpyDefault) != hipSuccess) {
    (void)hipGetLastError();
    return fail(SSD_E_INVAL, "prefix pointer not readable");
  }
  ssd_status cs = check_tokens_host(host.data(), host.size(), 0, m->dm.V, "prefix");
  if (cs != SSD_OK) return cs;
  ssd_session* s = nullptr;
  ssd_status st = create_session(m, B, P, max_ctx, max_block, stream ? (hipStream_t)stream : m->stream, &s);
  if (st != SSD_OK) return st;
  try {
    HIPCHK(hipMemcpyAsync(s->tok, host.data(), host.size() * 4, hipMemcpyHostToDevice, s->stream));
    prefill_pass(s);
    fwd_abort_fetch(s);
    HIPCHK(hipStreamSynchronize(s->stream));
    fwd_abort_check(s);
  } catch (HipError& e) {
    delete s;
    m->poisoned = true;
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  *out = s;
  return SSD_OK;
}

}  // extern "C"

// ---------------- spatial draft head ----------------
// Per-call device workspace of a draft head run: staging of the inputs, the
// activations of its four GEMMs (split bf16 planes), the x^2 partial sums, the
// draft logits, the split-K partials and their arrival counters.
struct HeadWork {
  int* tok = nullptr;      // [R]
  int* out = nullptr;      // [R]
  int* f0 = nullptr;       // one zero: the epilogues' block-start lookup
  float* hin = nullptr;    // [R][d]
  void* z = nullptr;       // [R][2d] split planes
  size_t z_plane = 0;
  float* x = nullptr;      // [R][d] fp32: u, then h_hat
  void* xn = nullptr;      // [R][d] split planes
  size_t xn_plane = 0;
  float* ssq = nullptr;    // [parts][rows]
  int ssq_cap = 0, rows = 0;
  void* hb = nullptr;      // [R][m] split planes
  size_t hb_plane = 0;
  float* logits = nullptr; // [R][V_img]
  float* gpart = nullptr;
  size_t gpart_cap = 0;
  unsigned* gcnt = nullptr;
  size_t gcnt_cap = 0;
};

struct ssd_draft_head {
  ssd_model* m;
  int d, mi, Rmax;
  bool poisoned = false;
  Allocs mem;
  void* w0;      // packed [d][2d]
  float* g;      // [d]
  void* w13;     // packed [2m][d], gate/up rows interleaved
  void* w2;      // packed [d][m]
  HeadWork work; // the head's own workspace (max_rows rows)
};

namespace {

// Enqueue one head on R rows of workspace w: hin [R][d] fp32 pre-norm states
// and tok [R] vocabulary ids (device).  Leaves the drafts (absolute image-code
// ids, lowest id among equal maxima) in w.out and the draft logits in w.logits.
void head_forward(ssd_draft_head* h, const HeadWork& w, int R, const float* hin, const int* tok, hipStream_t st) {
  ssd_model* m = h->m;
  const Dims& dm = m->dm;
  const int d = h->d, mi = h->mi;
  fill_u32((unsigned*)w.x, (size_t)R * d, 0u, st);  // u accumulates onto zero
  EpiArgs base{};
  base.Kblk = w.rows;  // every row is block position t of "sequence" 0
  base.f = w.f0;
  base.ssq_ld = w.rows;
  base.ssq_step = 1;
  base.inv_d = 1.0f / (float)d;
  base.eps = dm.eps;
  base.Hq = dm.Hq;
  base.Hkv = dm.Hkv;
  base.D = dm.D;
  base.x = w.x;
  base.xn = w.xn;
  base.xn_plane = w.xn_plane;
  base.ssq_out = w.ssq;
  base.ssq_out_ld = w.rows;
  base.h = w.hb;
  base.h_plane = w.hb_plane;
  base.logits = w.logits;
  if (!dm.bf16) {
    // fp32 models: plain fp32 GEMMs, one row sum of squares per norm
    draft_input_f32(hin, (const float*)m->emb, tok, R, d, (float*)w.z, st);
    EpiArgs e = base;
    e.kind = EPI_RESID;  // u = W0 [h; e]; n = g * u
    e.gnext = h->g;
    e.ld = d;
    gemm_f32((const float*)h->w0, d, 2 * d, (const float*)w.z, 2 * d, R, e, st);
    norm_rows_f32(w.x, R, d, nullptr, nullptr, w.ssq, st);
    e = base;
    e.kind = EPI_SWIGLU;  // SwiGLU(n / rms(u))
    e.ssq = w.ssq;
    e.ssq_parts = 1;
    e.ld = mi;
    gemm_f32((const float*)h->w13, 2 * mi, d, (const float*)w.xn, d, R, e, st);
    e = base;
    e.kind = EPI_RESID;  // h_hat = u + W2 (...); n = g_f * h_hat
    e.gnext = m->gf;
    e.ld = d;
    gemm_f32((const float*)h->w2, d, mi, (const float*)w.hb, mi, R, e, st);
    norm_rows_f32(w.x, R, d, nullptr, nullptr, w.ssq, st);
    e = base;
    e.kind = EPI_LOGITS;
    e.ssq = w.ssq;
    e.ssq_parts = 1;
    e.ld = dm.Vimg;
    gemm_f32((const float*)m->wlm, dm.Vimg, d, (const float*)w.xn, d, R, e, st);
  } else {
    draft_input(hin, m->emb, tok, R, d, w.z, w.z_plane, st);
    const int X = m->xcd;
    auto plan = [&](int N, int K) {
      GemmPlan p = gemm_plan_bf16(R, N, K, X);
      if (gemm_partials_floats(p, R) > w.gpart_cap || (size_t)gemm_counters(p) > w.gcnt_cap ||
          (N == d && p.n_fb > w.ssq_cap))
        throw HipError{hipErrorInvalidValue, "GEMM plan exceeds the draft head's workspace"};
      return p;
    };
    // u = W0 [h; e]; n = g * u (and the parts of sum u^2)
    GemmPlan p0 = plan(d, 2 * d);
    EpiArgs e = base;
    e.kind = EPI_RESID;
    e.gnext = h->g;
    e.ld = d;
    gemm_bf16(p0, h->w0, d, 2 * d, w.z, w.z_plane, 2 * d, R, e, w.gpart, w.gcnt, st);
    // SwiGLU(n / rms(u))
    GemmPlan p1 = plan(2 * mi, d);
    e = base;
    e.kind = EPI_SWIGLU;
    e.ssq = w.ssq;
    e.ssq_parts = p0.n_fb;
    e.ld = mi;
    gemm_bf16(p1, h->w13, 2 * mi, d, w.xn, w.xn_plane, d, R, e, w.gpart, w.gcnt, st);
    // h_hat = u + W2 (...); n = g_f * h_hat for the output layer
    GemmPlan p2 = plan(d, mi);
    e = base;
    e.kind = EPI_RESID;
    e.gnext = m->gf;
    e.ld = d;
    gemm_bf16(p2, h->w2, d, mi, w.hb, w.hb_plane, mi, R, e, w.gpart, w.gcnt, st);
    // GenHead(RMSNorm(h_hat)) over the image codes
    GemmPlan p3 = plan(dm.Vimg, d);
    e = base;
    e.kind = EPI_LOGITS;
    e.ssq = w.ssq;
    e.ssq_parts = p2.n_fb;
    e.ld = dm.Vimg;
    gemm_bf16(p3, m->wlm, dm.Vimg, d, w.xn, w.xn_plane, d, R, e, w.gpart, w.gcnt, st);
  }
  first_token(R, dm.Vimg, dm.img_lo, w.logits, SSD_GREEDY, 0, 1.0, 0, nullptr, w.out, 1, st);
  HIPCHK(hipGetLastError());
}

}  // namespace

extern "C" {

int64_t ssd_draft_head_numel(const ssd_model* m, int32_t mi) {
  if (!m || mi <= 0) return -1;
  const int64_t d = m->dm.d;
  return 2 * d * d + d + 3 * (int64_t)mi * d;
}

ssd_status ssd_draft_head_init(ssd_model* m, int32_t mi, const void* weights, int32_t max_rows,
                               ssd_draft_head** out) {
  g_err.clear();
  if (!m || !weights || !out) return fail(SSD_E_INVAL, "NULL argument");
  *out = nullptr;
  if (m->poisoned) return fail(SSD_E_STATE, "model is poisoned by an earlier device error");
  const Dims& dm = m->dm;
  if (mi <= 0 || mi % 256 != 0 || mi > (1 << 16)) return fail(SSD_E_INVAL, "m must be a positive multiple of 256");
  if (max_rows < 1 || max_rows > (1 << 16)) return fail(SSD_E_INVAL, "max_rows must be in [1, 65536]");
  auto* h = new ssd_draft_head();
  h->m = m;
  h->d = dm.d;
  h->mi = mi;
  h->Rmax = max_rows;
  const int d = dm.d;
  const size_t R = max_rows;
  hipStream_t st = m->stream;
  try {
    Allocs tmp;
    const size_t max_seg = std::max({(size_t)d * 2 * d, (size_t)2 * mi * d, (size_t)d * mi});
    uint16_t* stage = tmp.get<uint16_t>(max_seg * (dm.bf16 ? 1 : 2));
    std::vector<int> map_id(std::max({2 * d, 2 * mi, d})), map_13(2 * mi);
    for (size_t n = 0; n < map_id.size(); ++n) map_id[n] = (int)n;
    for (int n = 0; n < 2 * mi; ++n) map_13[n] = (n % 2 == 0) ? n / 2 : mi + n / 2;
    int* d_id = tmp.get<int>(map_id.size());
    int* d_13 = tmp.get<int>(map_13.size());
    HIPCHK(hipMemcpy(d_id, map_id.data(), map_id.size() * 4, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(d_13, map_13.data(), map_13.size() * 4, hipMemcpyHostToDevice));
    const uint16_t* src = (const uint16_t*)weights;
    if (!dm.bf16) {
      // fp32 models: row-major fp32 weights, gate/up rows interleaved
      const float* sf = (const float*)weights;
      auto copy = [&](size_t off, size_t n) -> float* {
        float* dst = h->mem.get<float>(n);
        HIPCHK(hipMemcpy(dst, sf + off, n * 4, hipMemcpyDefault));
        return dst;
      };
      size_t off = 0;
      h->w0 = copy(off, (size_t)d * 2 * d);
      off += (size_t)d * 2 * d;
      h->g = copy(off, d);
      off += d;
      HIPCHK(hipMemcpy(stage, sf + off, (size_t)2 * mi * d * 4, hipMemcpyDefault));
      h->w13 = h->mem.get<float>((size_t)2 * mi * d);
      gather_rows_f32((const float*)stage, d_13, 2 * mi, d, (float*)h->w13, st);
      HIPCHK(hipGetLastError());
      HIPCHK(hipStreamSynchronize(st));
      off += (size_t)2 * mi * d;
      h->w2 = copy(off, (size_t)d * mi);
    }
    auto pack = [&](size_t off, int N, int K, const int* map) -> void* {
      HIPCHK(hipMemcpy(stage, src + off, (size_t)N * K * 2, hipMemcpyDefault));
      void* dst = h->mem.get<char>((size_t)N * K * 2);
      pack_bf16_tiles(stage, map, N, K, dst, st);
      HIPCHK(hipGetLastError());
      HIPCHK(hipStreamSynchronize(st));
      return dst;
    };
    size_t off = 0;
    if (dm.bf16) h->w0 = pack(off, d, 2 * d, d_id);
    off += (size_t)d * 2 * d;
    if (dm.bf16) {
      std::vector<uint16_t> hb(d);
      HIPCHK(hipMemcpy(hb.data(), src + off, (size_t)d * 2, hipMemcpyDefault));
      std::vector<float> hf(d);
      for (int i = 0; i < d; ++i) {
        uint32_t u = (uint32_t)hb[i] << 16;
        std::memcpy(&hf[i], &u, 4);
      }
      h->g = h->mem.get<float>(d);
      HIPCHK(hipMemcpy(h->g, hf.data(), (size_t)d * 4, hipMemcpyHostToDevice));
    }
    off += d;
    if (dm.bf16) {
      h->w13 = pack(off, 2 * mi, d, d_13);
      off += (size_t)2 * mi * d;
      h->w2 = pack(off, d, mi, d_id);
    }
    // workspaces for every plan a run of up to max_rows rows can meet
    size_t gpart = 0, gcnt = 0;
    int parts = 1;
    for (int Mc : gemm_row_classes()) {
      if (!dm.bf16) break;
      for (auto nk : {std::make_pair(d, 2 * d), std::make_pair(2 * mi, d), std::make_pair(d, mi),
                      std::make_pair(dm.Vimg, d)}) {
        GemmPlan p = gemm_plan_bf16(Mc, nk.first, nk.second, 0);
        gpart = std::max(gpart, gemm_partials_floats(p, Mc));
        gcnt = std::max(gcnt, (size_t)gemm_counters(p));
        if (nk.first == d) parts = std::max(parts, std::max(p.n_fb, gemm_max_parts(d)));
      }
    }
    HeadWork& w = h->work;
    w.rows = (int)R;
    w.gpart_cap = gpart;
    w.gpart = h->mem.get<float>(gpart);
    w.gcnt_cap = gcnt;
    w.gcnt = h->mem.get<unsigned>(gcnt);
    w.ssq_cap = parts;
    w.ssq = h->mem.get<float>((size_t)parts * R);
    w.tok = h->mem.get<int>(R);
    w.out = h->mem.get<int>(R);
    w.f0 = h->mem.get<int>(1);
    w.hin = h->mem.get<float>(R * d);
    w.z_plane = R * 2 * d;
    w.z = h->mem.get<char>(R * 2 * d * 4);
    w.x = h->mem.get<float>(R * d);
    w.xn_plane = R * d;
    w.xn = h->mem.get<char>(R * d * 4);
    w.hb_plane = R * mi;
    w.hb = h->mem.get<char>(R * mi * 4);
    w.logits = h->mem.get<float>(R * dm.Vimg);
    fill_u32(w.gcnt, gcnt, 0u, st);
    fill_u32((unsigned*)w.f0, 1, 0u, st);
    HIPCHK(hipGetLastError());
    HIPCHK(hipStreamSynchronize(st));
  } catch (HipError& e) {
    delete h;
    if (e.e == hipErrorOutOfMemory || std::string(e.what) == "hipMalloc")
      return fail(SSD_E_OOM, "device allocation failed (%s)", hipGetErrorString(e.e));
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  *out = h;
  return SSD_OK;
}

ssd_status ssd_draft_head_run(ssd_draft_head* h, int32_t R, const float* hs, const int32_t* tokens, int32_t* drafts,
                              float* logits_out) {
  g_err.clear();
  if (!h || !hs || !tokens || !drafts) return fail(SSD_E_INVAL, "NULL argument");
  if (h->poisoned || h->m->poisoned) return fail(SSD_E_STATE, "draft head or model is poisoned");
  if (R < 1 || R > h->Rmax) return fail(SSD_E_INVAL, "R = %d outside [1, max_rows = %d]", R, h->Rmax);
  ssd_model* m = h->m;
  const Dims& dm = m->dm;
  const int d = h->d;
  if (!is_device_ptr(tokens)) {
    ssd_status cs = check_tokens_host(tokens, (size_t)R, 0, dm.V, "tokens");
    if (cs != SSD_OK) return cs;
  }
  const bool host_out = !is_device_ptr(drafts) || (logits_out && !is_device_ptr(logits_out));
  hipStream_t st = m->stream;
  try {
    const HeadWork& w = h->work;
    HIPCHK(hipMemcpyAsync(w.hin, hs, (size_t)R * d * 4, hipMemcpyDefault, st));
    HIPCHK(hipMemcpyAsync(w.tok, tokens, (size_t)R * 4, hipMemcpyDefault, st));
    head_forward(h, w, R, w.hin, w.tok, st);
    HIPCHK(hipMemcpyAsync(drafts, w.out, (size_t)R * 4, hipMemcpyDefault, st));
    if (logits_out) HIPCHK(hipMemcpyAsync(logits_out, w.logits, (size_t)R * dm.Vimg * 4, hipMemcpyDefault, st));
    if (host_out) HIPCHK(hipStreamSynchronize(st));
  } catch (HipError& e) {
    h->poisoned = true;
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  return SSD_OK;
}

ssd_status ssd_draft_head_run_noalloc(ssd_draft_head* h, int32_t R, const float* hs, const int32_t* tokens,
                                      int32_t* drafts, float* logits_out) {
  g_err.clear();
  if (!h || !hs || !tokens || !drafts) return fail(SSD_E_INVAL, "NULL argument");
  if (h->poisoned || h->m->poisoned) return fail(SSD_E_STATE, "draft head or model is poisoned");
  if (R < 1 || R > h->Rmax) return fail(SSD_E_INVAL, "R = %d outside [1, max_rows = %d]", R, h->Rmax);
  if (!is_device_ptr(hs) || !is_device_ptr(tokens) || !is_device_ptr(drafts) ||
      (logits_out && !is_device_ptr(logits_out)))
    return fail(SSD_E_INVAL, "the allocation-free run takes device arrays only");
  ssd_model* m = h->m;
  if (!m->scratch) return fail(SSD_E_STATE, "the static workspace's device address is unknown");
  const Dims& dm = m->dm;
  const int d = h->d, mi = h->mi;
  // carve this call's workspace out of the static array: every region 256-byte aligned
  size_t gpart = 0, gcnt = 0;
  int parts = 1;
  if (dm.bf16) {
    const std::pair<int, int> nk[4] = {{d, 2 * d}, {2 * mi, d}, {d, mi}, {dm.Vimg, d}};
    for (const auto& p : nk) {
      GemmPlan pl = gemm_plan_bf16(R, p.first, p.second, m->xcd);
      gpart = std::max(gpart, gemm_partials_floats(pl, R));
      gcnt = std::max(gcnt, (size_t)gemm_counters(pl));
      if (p.first == d) parts = std::max(parts, pl.n_fb);
    }
  }
  const size_t r = (size_t)R;
  const size_t sz[12] = {gcnt * 4, 4, r * 4, r * 4, r * d * 4, r * 2 * d * 4, r * d * 4, r * d * 4,
                         (size_t)parts * r * 4, r * mi * 4, r * dm.Vimg * 4, gpart * 4};
  size_t off[12], need = 0;
  for (int i = 0; i < 12; ++i) {
    off[i] = need;
    need += (sz[i] + 255) & ~(size_t)255;
  }
  if (need > NOALLOC_SCRATCH_BYTES)
    return fail(SSD_E_INVAL, "R = %d rows need %zu bytes of workspace; the static workspace holds %zu", R, need,
                NOALLOC_SCRATCH_BYTES);
  char* base = (char*)m->scratch;
  HeadWork w;
  w.rows = R;
  w.gcnt = (unsigned*)(base + off[0]);
  w.gcnt_cap = gcnt;
  w.f0 = (int*)(base + off[1]);
  w.tok = (int*)(base + off[2]);
  w.out = (int*)(base + off[3]);
  w.hin = (float*)(base + off[4]);
  w.z = base + off[5];
  w.z_plane = r * 2 * d;
  w.x = (float*)(base + off[6]);
  w.xn = base + off[7];
  w.xn_plane = r * d;
  w.ssq = (float*)(base + off[8]);
  w.ssq_cap = parts;
  w.hb = base + off[9];
  w.hb_plane = r * mi;
  w.logits = (float*)(base + off[10]);
  w.gpart = (float*)(base + off[11]);
  w.gpart_cap = gpart;
  hipStream_t st = m->stream;
  try {
    // the array keeps the last call's contents: counters and the block-start lookup start at zero
    fill_u32(w.gcnt, gcnt, 0u, st);
    fill_u32((unsigned*)w.f0, 1, 0u, st);
    HIPCHK(hipMemcpyAsync(w.hin, hs, r * d * 4, hipMemcpyDeviceToDevice, st));
    HIPCHK(hipMemcpyAsync(w.tok, tokens, r * 4, hipMemcpyDeviceToDevice, st));
    head_forward(h, w, R, w.hin, w.tok, st);
    HIPCHK(hipMemcpyAsync(drafts, w.out, r * 4, hipMemcpyDeviceToDevice, st));
    if (logits_out) HIPCHK(hipMemcpyAsync(logits_out, w.logits, r * dm.Vimg * 4, hipMemcpyDeviceToDevice, st));
  } catch (HipError& e) {
    h->poisoned = true;
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  return SSD_OK;
}

void ssd_free_draft_head(ssd_draft_head* h) {
  if (!h) return;
  (void)hipStreamSynchronize(h->m->stream);
  delete h;
}

ssd_status ssd_profile(ssd_model* m, int32_t enable) {
  if (!m) return fail(SSD_E_INVAL, "NULL model");
  try {
    HIPCHK(hipStreamSynchronize(m->stream));
    m->prof.flush();
    m->prof.on = enable != 0;
  } catch (HipError& e) {
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  return SSD_OK;
}

ssd_status ssd_profile_read(ssd_model* m, double* ms, int64_t* launches, double* bytes, double* flops,
                            int32_t reset) {
  if (!m) return fail(SSD_E_INVAL, "NULL model");
  try {
    HIPCHK(hipStreamSynchronize(m->stream));
    m->prof.flush();
  } catch (HipError& e) {
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  for (int c = 0; c < Prof::NCLS; ++c) {
    if (ms) ms[c] = m->prof.ms[c];
    if (launches) launches[c] = m->prof.n[c];
    if (bytes) bytes[c] = m->prof.bytes[c];
    if (flops) flops[c] = m->prof.flops[c];
    if (reset) {
      m->prof.ms[c] = 0;
      m->prof.n[c] = 0;
      m->prof.bytes[c] = 0;
      m->prof.flops[c] = 0;
    }
  }
  return SSD_OK;
}

ssd_status ssd_get_carry(ssd_session* s, float* carry_out) {
  if (!s || !carry_out) return fail(SSD_E_INVAL, "NULL argument");
  if (s->poisoned) return fail(SSD_E_STATE, "session is poisoned");
  const float* src = s->carry;
  if (s->cfg) {
    cfg_mix(s->Bi, 0, s->dm.Vimg, s->cfg_w, nullptr, s->carry, nullptr, s->mcarry, s->stream);
    src = s->mcarry;
  }
  if (hipGetLastError() != hipSuccess ||
      hipMemcpyAsync(carry_out, src, (size_t)s->Bi * s->dm.Vimg * 4, hipMemcpyDefault, s->stream) != hipSuccess ||
      hipStreamSynchronize(s->stream) != hipSuccess) {
    s->poisoned = true;
    return fail(SSD_E_DEVICE, "copy of the carry failed");
  }
  return SSD_OK;
}

ssd_status ssd_session_set_cfg(ssd_session* s, float weight) {
  g_err.clear();
  if (!s) return fail(SSD_E_INVAL, "NULL session");
  if (s->poisoned) return fail(SSD_E_STATE, "session is poisoned");
  if (!std::isfinite(weight)) return fail(SSD_E_INVAL, "guidance weight must be finite");
  if (!s->cfg) {
    if (s->B % 2) return fail(SSD_E_INVAL, "guidance pairs sequences: B = %d is odd", s->B);
    try {
      if (!s->mlog) {
        s->mlog = s->mem.get<float>((size_t)(s->B / 2) * s->Kmax * s->dm.Vimg);
        s->mcarry = s->mem.get<float>((size_t)(s->B / 2) * s->dm.Vimg);
      }
    } catch (HipError& e) {
      return fail(SSD_E_OOM, "%s: %s", e.what, hipGetErrorString(e.e));
    }
    s->cfg = true;
    s->Bi = s->B / 2;
  }
  s->cfg_w = weight;
  return SSD_OK;
}

ssd_status ssd_verify_step(ssd_session* s, int32_t K, int32_t* tokens, const float* ref_logits,
                           const ssd_verify_params* prm, uint8_t* accept_mask, int32_t* accept_count,
                           int32_t* frontier, float* logits_out, float* h_pre_out) {
  g_err.clear();
  if (!s || !tokens || !prm) return fail(SSD_E_INVAL, "NULL argument");
  if (s->poisoned) return fail(SSD_E_STATE, "session is poisoned by an earlier device error");
  const Dims& dm = s->dm;
  const int B = s->B;
  const int nb = s->Bi;  // rows of every per-image argument (B, or B / 2 when guided)
  if (K < 1 || K > s->Kmax) return fail(SSD_E_INVAL, "K = %d outside [1, max_block = %d]", K, s->Kmax);
  if (prm->rule < SSD_GREEDY || prm->rule > SSD_ACCEPT_REJECT) return fail(SSD_E_INVAL, "unknown rule");
  if (!(prm->temperature > 0.0)) return fail(SSD_E_INVAL, "temperature must be > 0");
  if (prm->n_fixed < 0 || prm->n_fixed > 1 || prm->n_fixed > K) return fail(SSD_E_INVAL, "n_fixed must be 0 or 1 (<= K)");
  if (prm->round >= 65536u) return fail(SSD_E_INVAL, "round must be < 65536");
  if (prm->truncate && (prm->commit || prm->rule != SSD_GREEDY))
    return fail(SSD_E_INVAL, "truncate needs rule SSD_GREEDY and commit = 0");
  if (prm->truncate && s->cfg) return fail(SSD_E_INVAL, "truncate is not available on a guided session");
  for (int b = 0; b < B; ++b)
    if (s->f[b] + K > s->max_ctx || s->f[b] + K >= (1 << 24))
      return fail(SSD_E_CAPACITY, "block [%d, %d) of sequence %d exceeds max_ctx", s->f[b], s->f[b] + K, b);
  const bool tok_dev = is_device_ptr(tokens);
  std::vector<int32_t> htok;
  if (!tok_dev) {
    ssd_status cs = check_tokens_host(tokens, (size_t)nb * K, dm.img_lo, dm.img_hi, "tokens");
    if (cs != SSD_OK) return cs;
  }
  const bool host_out = (!tok_dev && !prm->commit) || (accept_mask && !is_device_ptr(accept_mask)) ||
                        (accept_count && !is_device_ptr(accept_count)) || (frontier && !is_device_ptr(frontier)) ||
                        (logits_out && !is_device_ptr(logits_out)) || (h_pre_out && !is_device_ptr(h_pre_out));
  hipStream_t st = s->stream;
  try {
    HIPCHK(hipMemcpyAsync(s->tok, tokens, (size_t)nb * K * 4, hipMemcpyDefault, st));
    // a guided image's block goes to both of its streams
    if (s->cfg) HIPCHK(hipMemcpyAsync(s->tok + (size_t)nb * K, s->tok, (size_t)nb * K * 4, hipMemcpyDeviceToDevice, st));
    if (ref_logits && !prm->commit)
    {
      // the caller's array may be host memory: stage it on the device first
      HIPCHK(hipMemcpyAsync(s->refstage, ref_logits, (size_t)nb * K * dm.Vimg * 4, hipMemcpyDefault, st));
      set_ref_rows(nb, K, K, dm.Vimg, s->refstage, s->d_f, s->ref, s->ref_flag, s->ring, 0, st);
    }
    const bool all_rows = !prm->commit || logits_out;
    run_forward(s, K, all_rows ? 0 : 1);
    // per-image scores: the pass's own logits, or the guided mix of the two streams
    const float* lg = s->logits;
    const float* cy = s->carry;
    if (s->cfg && all_rows) {
      cfg_mix(nb, K, dm.Vimg, s->cfg_w, s->logits, s->carry, s->mlog, s->mcarry, st);
      lg = s->mlog;
      cy = s->mcarry;
    }
    if (logits_out) HIPCHK(hipMemcpyAsync(logits_out, lg, (size_t)nb * K * dm.Vimg * 4, hipMemcpyDefault, st));
    if (h_pre_out) HIPCHK(hipMemcpyAsync(h_pre_out, s->x, (size_t)nb * K * dm.d * 4, hipMemcpyDefault, st));
    if (prm->commit) {
      commit_update(B, all_rows ? K : -K, dm.Vimg, s->logits, s->carry, s->d_f, s->ref_flag, s->ring, st);
      for (int b = 0; b < B; ++b) s->f[b] += K;
    } else {
      fill_u32((unsigned*)s->cnt, nb, 0u, st);
      SelectArgs a{};
      a.rule = prm->rule;
      a.top_k = prm->top_k;
      a.temperature = prm->temperature;
      a.seed = prm->seed;
      a.round = prm->round;
      a.n_fixed = prm->n_fixed;
      a.K = K;
      a.B = nb;
      a.Vimg = dm.Vimg;
      a.img_lo = dm.img_lo;
      a.truncate = prm->truncate;
      a.f = s->d_f;
      a.tokens = s->tok;
      a.logits = lg;
      a.carry = cy;
      a.ref = s->ref;
      a.ref_flag = s->ref_flag;
      a.ring = s->ring;
      a.accept = s->acc;
      a.count = s->cnt;
      a.amax = s->amax;
      select_tokens(a, st);
      if (prm->truncate) truncate_finalize(a, s->d_f, st);
      HIPCHK(hipGetLastError());
      HIPCHK(hipMemcpyAsync(tokens, s->tok, (size_t)nb * K * 4, hipMemcpyDefault, st));
      if (accept_mask) HIPCHK(hipMemcpyAsync(accept_mask, s->acc, (size_t)nb * K, hipMemcpyDefault, st));
      if (accept_count) HIPCHK(hipMemcpyAsync(accept_count, s->cnt, (size_t)nb * 4, hipMemcpyDefault, st));
      if (prm->truncate) {
        HIPCHK(hipMemcpyAsync(s->f.data(), s->d_f, (size_t)B * 4, hipMemcpyDeviceToHost, st));
        fwd_abort_fetch(s);
        HIPCHK(hipStreamSynchronize(st));
        fwd_abort_check(s);
      }
    }
    if (frontier) HIPCHK(hipMemcpyAsync(frontier, s->d_f, (size_t)nb * 4, hipMemcpyDefault, st));
    if (host_out) {
      fwd_abort_fetch(s);
      HIPCHK(hipStreamSynchronize(st));
      fwd_abort_check(s);
      s->m->prof.flush();
    }
  } catch (HipError& e) {
    s->poisoned = true;
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  return SSD_OK;
}

// ---------------- image schedule driver ----------------
namespace {

struct Op {
  int kind;  // 0 verify, 1 commit, 2 horizontal draft (src, K heads), 3 vertical draft (row src, K rows)
  int start, K, nf, rnd;
  int rib;   // verify: rounds of this block before this one since it was drafted
};

// pass plan of one image (mirrors the schedule documented in ssd.h)
// eol: verify/commit blocks are in sequence positions (row y starts at
// y * (W + 1)) and a block that completes a row includes its end-of-line slot
std::vector<Op> make_plan(int H, int W, int k_h, int h_rounds, int k_v, int b, int i, bool eol = false) {
  std::vector<Op> ops;
  int rnd = 0;
  const int RW = eol ? W + 1 : W, tail = eol ? 1 : 0;
  auto verify = [&](int start, int K, int nf, int count) {
    for (int c = 0; c < count; ++c) ops.push_back(Op{0, start, K, nf, rnd++, c});
  };
  bool first = true;
  for (int s = 1; s < W;) {
    int e = std::min(s + k_h, W);
    const int t = e == W ? tail : 0;
    if (first) {
      ops.push_back(Op{2, 0, e - 1, 0, 0});
      verify(0, e + t, 1, h_rounds);
      ops.push_back(Op{1, 0, e + t, 0, 0});
      first = false;
    } else {
      ops.push_back(Op{2, s - 1, e - s, 0, 0});
      verify(s, e - s + t, 0, h_rounds);
      ops.push_back(Op{1, s, e - s + t, 0, 0});
    }
    s = e;
  }
  if (W == 1) ops.push_back(Op{1, 0, 1 + tail, 0, 0});
  for (int y = 1; y < H;) {
    int m = std::min(k_v, H - y);
    ops.push_back(Op{3, y - 1, m, 0, 0});
    verify(y * RW, m * RW, 0, b);
    ops.push_back(Op{1, y * RW, RW, 0, 0});
    for (int j = 1; j < m; ++j) {
      verify((y + j) * RW, (m - j) * RW, 0, i);
      ops.push_back(Op{1, (y + j) * RW, RW, 0, 0});
    }
    y += m;
  }
  return ops;
}

}  // namespace

namespace {

// Draft source of an image decode: a planted table (drafts, optional draft
// logits) or spatial heads (horizontal heads for offsets +1.., vertical heads
// for rows +1..).
struct DraftSource {
  const int32_t* drafts = nullptr;
  const float* draft_logits = nullptr;
  ssd_draft_head* const* hh = nullptr;
  int nh = 0;
  ssd_draft_head* const* vh = nullptr;
  int nv = 0;
  // planting (ssd_plant_image): drafts made left to right against the decode's own argmax
  const uint8_t* keep = nullptr;
  const int32_t* repl = nullptr;
  int32_t* table = nullptr;
};

ssd_status decode_impl(ssd_model* m, const ssd_schedule* sc, int32_t B, int32_t P, const int32_t* prefix,
                       const DraftSource& src, int32_t* out_tokens, ssd_stats* stats, void* stream) {
  const auto t_call = std::chrono::steady_clock::now();
  const int32_t* drafts = src.drafts;
  const float* draft_logits = src.draft_logits;
  const bool heads = src.hh != nullptr || src.vh != nullptr;
  const bool plant = src.keep != nullptr;
  if (m->poisoned) return fail(SSD_E_STATE, "model is poisoned by an earlier device error");
  const Dims& dm = m->dm;
  const int H = sc->grid_h, W = sc->grid_w;
  if (H < 1 || W < 1 || B < 1 || B >= (1 << 20) || P < 1) return fail(SSD_E_INVAL, "bad grid, batch or prefix size");
  if ((int64_t)H * W >= (1 << 24)) return fail(SSD_E_INVAL, "image too large");
  if (sc->k_h < 1 || sc->h_rounds < 0 || sc->k_v < 1 || sc->b_rounds < 0 || sc->i_rounds < 0)
    return fail(SSD_E_INVAL, "bad schedule");
  if (sc->rule < SSD_GREEDY || sc->rule > SSD_ACCEPT_REJECT || !(sc->temperature > 0.0))
    return fail(SSD_E_INVAL, "bad rule or temperature");
  if ((sc->cfg != 0 && sc->cfg != 1) || (sc->cfg && !std::isfinite(sc->cfg_weight)))
    return fail(SSD_E_INVAL, "cfg must be 0 or 1 with a finite weight");
  if (sc->cfg && B >= (1 << 19)) return fail(SSD_E_INVAL, "bad batch size");
  const int Bs = sc->cfg ? 2 * B : B;  // sequences: a guided image has two streams
  if (sc->eol != 0 && sc->eol != 1) return fail(SSD_E_INVAL, "eol must be 0 or 1");
  const bool eol = sc->eol == 1;
  if (eol && (sc->eol_id < 0 || sc->eol_id >= dm.V)) return fail(SSD_E_INVAL, "eol_id outside the vocabulary");
  if (sc->truncate != 0 && sc->truncate != 1) return fail(SSD_E_INVAL, "truncate must be 0 or 1");
  const bool trunc = sc->truncate == 1;
  if (trunc) {
    if (sc->rule != SSD_GREEDY) return fail(SSD_E_INVAL, "the strict decode needs rule SSD_GREEDY");
    if (sc->cfg || eol || heads) return fail(SSD_E_INVAL, "the strict decode takes no guidance, row ends or heads");
    if (sc->trunc_block < 2 || sc->trunc_block > 4096) return fail(SSD_E_INVAL, "trunc_block must be in [2, 4096]");
  }
  if (plant && (sc->cfg || eol || draft_logits || heads))
    return fail(SSD_E_INVAL, "planting takes no guidance, row ends, draft logits or heads");
  const int N = H * W;
  const int RW = eol ? W + 1 : W;  // sequence positions per image row
  // working row of an image: its sequence positions, plus one block of slack
  // for the strict decode (blocks past the last token read it)
  const int NS = trunc ? N + sc->trunc_block : H * RW;
  const int Lmax = P + NS;
  if (Lmax >= (1 << 24)) return fail(SSD_E_INVAL, "image too large");
  if (!dm.bf16 && Lmax > 4096) return fail(SSD_E_INVAL, "fp32 models support P + image positions <= 4096");
  std::vector<Op> ops;
  if (!trunc) ops = make_plan(H, W, sc->k_h, sc->h_rounds, sc->k_v, sc->b_rounds, sc->i_rounds, eol);
  if (sc->separate_commit != 0 && sc->separate_commit != 1) return fail(SSD_E_INVAL, "separate_commit must be 0 or 1");
  // fuse[i]: commit op i runs inside the pass of the verify round right after it
  // (adjacent block, nothing fixed at its start, no head drafting in between:
  // drafting needs the committed states first)
  std::vector<char> fuse(ops.size(), 0);
  int Kmax = trunc ? sc->trunc_block : 1;
  int nverify = 0;
  for (size_t i = 0; i < ops.size(); ++i) {
    const Op& o = ops[i];
    if (o.kind <= 1) Kmax = std::max(Kmax, o.K);
    nverify += o.kind == 0;
    if (o.kind != 1 || sc->separate_commit) continue;
    size_t j = i + 1;
    while (j < ops.size() && ops[j].kind >= 2 && !heads) ++j;
    if (j < ops.size() && ops[j].kind == 0 && ops[j].nf == 0 && ops[j].start == o.start + o.K) {
      fuse[i] = 1;
      Kmax = std::max(Kmax, o.K + ops[j].K);
    }
  }
  if (heads) {
    // every head the plan calls must exist, belong to this model and hold its rows
    for (const Op& o : ops) {
      if (o.kind < 2) continue;
      const bool hor = o.kind == 2;
      const int need = hor ? B : B * W;
      for (int j = 0; j < o.K; ++j) {
        ssd_draft_head* h = j < (hor ? src.nh : src.nv) ? (hor ? src.hh : src.vh)[j] : nullptr;
        if (!h) return fail(SSD_E_INVAL, "the schedule needs %s head %d", hor ? "horizontal" : "vertical", j + 1);
        if (h->m != m) return fail(SSD_E_INVAL, "a draft head belongs to another model");
        if (h->poisoned) return fail(SSD_E_STATE, "a draft head is poisoned");
        if (h->Rmax < need) return fail(SSD_E_INVAL, "a %s head drafts %d rows per call here; its max_rows is %d",
                                        hor ? "horizontal" : "vertical", need, h->Rmax);
      }
    }
  }
  if (nverify >= 65536) return fail(SSD_E_INVAL, "more than 65535 verify rounds");
  std::vector<int32_t> hpre((size_t)Bs * P), hdr((size_t)B * N, dm.img_lo);
  std::vector<uint8_t> hkeep;
  if (hipMemcpy(hpre.data(), prefix, hpre.size() * 4, hipMemcpyDefault) != hipSuccess ||
      (!heads && !plant && hipMemcpy(hdr.data(), drafts, hdr.size() * 4, hipMemcpyDefault) != hipSuccess)) {
    (void)hipGetLastError();
    return fail(SSD_E_INVAL, "prefix or drafts not readable");
  }
  if (plant) {
    hkeep.resize((size_t)B * N);
    if (hipMemcpy(hkeep.data(), src.keep, hkeep.size(), hipMemcpyDefault) != hipSuccess ||
        hipMemcpy(hdr.data(), src.repl, hdr.size() * 4, hipMemcpyDefault) != hipSuccess) {
      (void)hipGetLastError();
      return fail(SSD_E_INVAL, "keep or repl not readable");
    }
    ssd_status rs = check_tokens_host(hdr.data(), hdr.size(), 0, dm.Vimg - 1, "repl");
    if (rs != SSD_OK) return rs;
    for (auto& v : hdr) v += dm.img_lo;  // the table before planting: the replacement codes as ids
  }
  ssd_status cs = check_tokens_host(hpre.data(), hpre.size(), 0, dm.V, "prefix");
  if (cs != SSD_OK) return cs;
  cs = check_tokens_host(hdr.data(), hdr.size(), dm.img_lo, dm.img_hi, "drafts");
  if (cs != SSD_OK) return cs;
  if (eol || trunc) {  // the working table holds sequence positions (row ends, or the strict decode's slack)
    std::vector<int32_t> seq((size_t)B * NS, eol ? sc->eol_id : dm.img_lo);
    if (eol) {
      for (size_t r = 0; r < (size_t)B * H; ++r) std::memcpy(&seq[r * RW], &hdr[r * W], (size_t)W * 4);
    } else {
      for (size_t b = 0; b < (size_t)B; ++b) std::memcpy(&seq[b * NS], &hdr[b * N], (size_t)N * 4);
    }
    hdr.swap(seq);
  }
  const hipStream_t call_st = stream ? (hipStream_t)stream : m->stream;
  // decode workspace, reused across calls of the same shape (a longer block bound serves shorter blocks)
  if (!m->dec || m->dec_B != Bs || m->dec_P != P || m->dec_L != Lmax || m->dec_K < Kmax) {
    if (m->dec) {
      ssd_session* old = m->dec;
      m->dec = nullptr;
      delete old;
    }
    ssd_session* s = nullptr;
    ssd_status st = create_session(m, Bs, P, Lmax, Kmax, call_st, &s);
    if (st != SSD_OK) return st;
    m->dec = s;
    m->dec_B = Bs;
    m->dec_P = P;
    m->dec_L = Lmax;
    m->dec_K = Kmax;
  }
  ssd_session* s = m->dec;
  s->stream = call_st;
  if (sc->cfg) {
    ssd_status gs = ssd_session_set_cfg(s, (float)sc->cfg_weight);
    if (gs != SSD_OK) return gs;
  } else {
    s->cfg = false;
    s->Bi = s->B;
  }
  hipStream_t st = s->stream;
  int64_t passes = 0, nv = 0, proposed = 0;
  int64_t prop_round[NCNT_ROUNDS] = {0};
  std::vector<int> hc((size_t)NCNT_ROUNDS * Bs, 0);  // accept counters [round][sequence]
  int64_t acc_trunc = 0;
  try {
    if (s->img_cap < B * NS) {
      s->img = s->mem.get<int>((size_t)B * NS);
      s->img_cap = B * NS;
    }
    const bool use_q = sc->rule == SSD_ACCEPT_REJECT && (draft_logits || heads);
    if (use_q && s->qtab_cap < (size_t)B * NS * dm.Vimg) {
      s->qtab = s->mem.get<float>((size_t)B * NS * dm.Vimg);
      s->qtab_cap = (size_t)B * NS * dm.Vimg;
    }
    if (heads && s->hs_cap < (size_t)B * N * dm.d) {
      s->hs = s->mem.get<float>((size_t)B * N * dm.d);
      s->hs_cap = (size_t)B * N * dm.d;
      s->hsrc = s->mem.get<float>((size_t)B * W * dm.d);
      s->tsrc = s->mem.get<int>((size_t)B * W);
    }
    if (plant) {
      if (s->plant_cap < (size_t)B * N) {
        s->pkeep = s->mem.get<unsigned char>((size_t)B * N);
        s->prepl = s->mem.get<int>((size_t)B * N);
        s->ptab = s->mem.get<int>((size_t)B * N);
        s->pactive = s->mem.get<int>((size_t)B);
        s->plant_cap = (size_t)B * N;
      }
      HIPCHK(hipMemcpyAsync(s->pkeep, hkeep.data(), hkeep.size(), hipMemcpyHostToDevice, st));
      HIPCHK(hipMemcpy2DAsync(s->ptab, (size_t)N * 4, hdr.data(), (size_t)NS * 4, (size_t)N * 4, B,
                              hipMemcpyHostToDevice, st));
      HIPCHK(hipMemcpy2DAsync(s->prepl, (size_t)N * 4, hdr.data(), (size_t)NS * 4, (size_t)N * 4, B,
                              hipMemcpyHostToDevice, st));
      add_i32(s->prepl, B * N, -dm.img_lo, st);  // back to code indices
    }
    HIPCHK(hipMemcpyAsync(s->img, hdr.data(), hdr.size() * 4, hipMemcpyHostToDevice, st));
    if (draft_logits)  // [B][H][W][V] into the sequence layout (end-of-line rows are never read)
      HIPCHK(hipMemcpy2DAsync(s->qtab, (size_t)RW * dm.Vimg * 4, draft_logits, (size_t)W * dm.Vimg * 4,
                              (size_t)W * dm.Vimg * 4, (size_t)B * H, hipMemcpyDefault, st));
    fill_u32((unsigned*)s->d_f, Bs, 0u, st);
    fill_u32((unsigned*)s->ref_flag, (size_t)Bs * s->ring, 0u, st);
    fill_u32((unsigned*)s->cnt, (size_t)NCNT_ROUNDS * Bs, 0u, st);
    for (int b = 0; b < Bs; ++b) s->f[b] = 0;
    HIPCHK(hipMemcpyAsync(s->tok, hpre.data(), hpre.size() * 4, hipMemcpyHostToDevice, st));
    prefill_pass(s);
    ++passes;
    const size_t rowb = (size_t)dm.d * 4;  // bytes of one state
    if (heads)  // the state that scores image token 0: the prompt's last (conditional streams)
      HIPCHK(hipMemcpy2DAsync(s->hs, (size_t)N * rowb, s->x + (size_t)(P - 1) * dm.d, (size_t)P * rowb, rowb, B,
                              hipMemcpyDeviceToDevice, st));
    // per-image scores: the streams' own logits, or their guided mix
    const float* lg = s->cfg ? s->mlog : s->logits;
    const float* cy = s->cfg ? s->mcarry : s->carry;
    if (s->cfg) cfg_mix(B, 0, dm.Vimg, s->cfg_w, nullptr, s->carry, nullptr, s->mcarry, st);
    first_token(B, dm.Vimg, dm.img_lo, cy, sc->rule, sc->top_k, sc->temperature, sc->seed, s->d_f, s->img, NS, st);
    SelectArgs a{};
    a.rule = sc->rule;
    a.top_k = sc->top_k;
    a.temperature = sc->temperature;
    a.seed = sc->seed;
    a.B = B;
    a.Vimg = dm.Vimg;
    a.img_lo = dm.img_lo;
    a.f = s->d_f;
    a.tokens = s->tok;
    a.logits = lg;
    a.carry = cy;
    a.ref = s->ref;
    a.ref_flag = s->ref_flag;
    a.ring = s->ring;
    a.accept = s->acc;
    a.count = s->cnt;
    a.amax = s->amax;
    a.eol_period = eol ? RW : 0;
    a.eol_base = P;
    // planting: the argmax of a logits row placed as a planted draft
    PlaceArgs pa{};
    pa.row_stride = dm.Vimg;
    pa.Vimg = dm.Vimg;
    pa.img_lo = dm.img_lo;
    pa.f = s->d_f;
    pa.P = P;
    pa.x_end = N;
    pa.img = s->img;
    pa.img_stride = NS;
    pa.keep = s->pkeep;
    pa.repl = s->prepl;
    pa.table = s->ptab;
    pa.next_tok = s->tok;
    // Move every frontier by delta (device and host mirror): the single-position
    // planting passes run at positions past the committed context.
    auto shift_f = [&](int delta) {
      add_i32(s->d_f, B, delta, st);
      for (int b = 0; b < B; ++b) s->f[b] += delta;
    };
    if (trunc) {
      // ---- strict greedy verification: blocks [pending, K-1 drafts] at each sequence's frontier ----
      const int K = sc->trunc_block;
      // the first pending token: the argmax of the prefill's carry (first_token above)
      std::vector<int> done(B, 0), fh(B), cnt_h(B);
      PlaceArgs pend{};
      pend.logits = s->carry;
      pend.row_stride = dm.Vimg;
      pend.Vimg = dm.Vimg;
      pend.img_lo = dm.img_lo;
      pend.f = s->d_f;
      pend.P = P;
      pend.x_end = NS;
      pend.img = s->img;
      pend.img_stride = NS;
      while (true) {
        int rem = 0;  // positions left after the pending token, over the live sequences
        for (int b = 0; b < B; ++b)
          if (done[b] < N - 1) rem = std::max(rem, N - done[b]);
        if (rem == 0) break;
        const int Kp = std::min(K, rem);
        if (plant) {
          // plant what this pass tests: positions after the pending token, left to
          // right, each from a single-position pass over its predecessor, while the
          // drafts so far are kept (the first replacement ends a sequence's planting)
          std::vector<int> act(B);
          for (int b = 0; b < B; ++b) act[b] = done[b] < N - 1;
          HIPCHK(hipMemcpy(s->pactive, act.data(), (size_t)B * 4, hipMemcpyHostToDevice));
          gather_block(s->img, NS, s->d_f, P, 1, B, s->tok, st);
          pa.active = s->pactive;
          pa.pos_off = 1;
          pa.logits = s->logits;
          int moved = 0;
          for (int j = 0; j + 1 < Kp; ++j) {
            if (j > 0) {
              shift_f(1);
              ++moved;
            }
            run_forward(s, 1, 1);
            place_argmax(pa, B, st);
            HIPCHK(hipMemcpyAsync(act.data(), s->pactive, (size_t)B * 4, hipMemcpyDeviceToHost, st));
            HIPCHK(hipStreamSynchronize(st));
            bool any = false;
            for (int b = 0; b < B; ++b) any |= act[b] != 0;
            if (!any) break;
          }
          shift_f(-moved);
          pa.active = nullptr;
        }
        gather_block(s->img, NS, s->d_f, P, Kp, B, s->tok, st);
        run_forward(s, Kp, 0);
        a.K = Kp;
        a.n_fixed = 1;
        a.round = 0;
        a.truncate = 1;
        a.count = s->cnt;
        select_tokens(a, st);
        truncate_finalize(a, s->d_f, st);  // f += 1 + accepted run; carry <- logits scoring the next pending
        place_argmax(pend, B, st);         // next pending token at the new frontier
        HIPCHK(hipMemcpyAsync(fh.data(), s->d_f, (size_t)B * 4, hipMemcpyDeviceToHost, st));
        HIPCHK(hipMemcpyAsync(cnt_h.data(), s->cnt, (size_t)B * 4, hipMemcpyDeviceToHost, st));
        fwd_abort_fetch(s);
        HIPCHK(hipStreamSynchronize(st));
        fwd_abort_check(s);
        ++passes;
        ++nv;
        bool freeze = false;
        for (int b = 0; b < B; ++b) {
          if (done[b] >= N - 1) {  // finished earlier: frozen at its last position
            fh[b] = P + N - 1;
            freeze = true;
            continue;
          }
          const int room = N - 1 - done[b];  // drafts of this pass inside the image
          const int n = std::min(cnt_h[b], room);
          acc_trunc += n;
          proposed += n + ((n < Kp - 1 && n < room) ? 1 : 0);
          done[b] = fh[b] - P;
          if (done[b] >= N - 1) {
            fh[b] = P + N - 1;
            freeze |= done[b] > N - 1;
            done[b] = N - 1;
          }
        }
        for (int b = 0; b < B; ++b) s->f[b] = fh[b];
        if (freeze) HIPCHK(hipMemcpy(s->d_f, fh.data(), (size_t)B * 4, hipMemcpyHostToDevice));
      }
      a.truncate = 0;
    }
    // the state of block offset k (pass rows of `rps` per sequence) scores sequence
    // position start + k + 1: kept under its image index when that is an image
    // position (a row end's state scores the next row's first token), one copy per
    // run of such offsets
    auto keep_states = [&](int start, int Kc, int rps) {
      for (int k = 0; heads && k < Kc;) {
        int q1 = start + k + 1;
        if (q1 >= NS || q1 % RW == W) {
          ++k;
          continue;
        }
        int len = 1;
        while (k + len < Kc && q1 + len < NS && (q1 + len) % RW != W) ++len;
        const int p1 = (q1 / RW) * W + q1 % RW;
        HIPCHK(hipMemcpy2DAsync(s->hs + (size_t)p1 * dm.d, (size_t)N * rowb, s->x + (size_t)k * dm.d,
                                (size_t)rps * rowb, (size_t)len * rowb, B, hipMemcpyDeviceToDevice, st));
        k += len;
      }
    };
    // planted drafts of image indexes [q0, q0 + n), left to right: the first from
    // the logits that score q0 (the carry, or a pass over the chosen but not yet
    // cached tokens before q0: a commit that runs inside the next verify pass, or
    // the first image token), each later one from a single-position pass over its
    // predecessor.  The KV slots these passes write lie inside the next verify
    // pass's block, which rewrites them before reading.
    auto plant_block = [&](int q0, int n) {
      const int x0 = s->f[0] - P;  // first image index not cached (equal for all sequences)
      const int Kc = q0 - x0;
      if (Kc < 0 || Kc > s->Kmax) throw HipError{hipErrorInvalidValue, "planting outside the plan"};
      if (Kc > 0) {
        HIPCHK(hipMemcpy2DAsync(s->tok, (size_t)Kc * 4, s->img + x0, (size_t)NS * 4, (size_t)Kc * 4, B,
                                hipMemcpyDeviceToDevice, st));
        run_forward(s, Kc, 1);
      }
      pa.logits = Kc > 0 ? s->logits : s->carry;
      pa.pos_off = Kc;
      place_argmax(pa, B, st);
      pa.logits = s->logits;
      pa.pos_off = 1;
      int moved = 0;
      for (int j = 1; j < n; ++j) {
        shift_f(Kc + j - 1 - moved);  // the pass reads the draft at image index q0 + j - 1
        moved = Kc + j - 1;
        run_forward(s, 1, 1);
        place_argmax(pa, B, st);
      }
      shift_f(-moved);
    };
    const Op* pending = nullptr;  // a commit waiting for the verify round it runs with
    for (size_t i = 0; i < ops.size(); ++i) {
      const Op& o = ops[i];
      if (o.kind >= 2) {
        if (plant) {
          if (o.kind == 2)
            plant_block(o.start + 1, o.K);
          else
            plant_block((o.start + 1) * W, o.K * W);
          continue;
        }
        if (!heads) continue;
        // heads draft from chosen tokens: [h; e] with h the state that scored each
        // (image indices for the states, sequence positions for the tokens)
        const bool hor = o.kind == 2;
        const int n_src = hor ? 1 : W;                 // source positions per image
        const int p0 = hor ? o.start : o.start * W;    // first source image index
        const int step = hor ? 1 : W;                  // offset of head j is j * step
        auto seq_of = [&](int p) { return (p / W) * RW + p % W; };
        HIPCHK(hipMemcpy2DAsync(s->hsrc, n_src * rowb, s->hs + (size_t)p0 * dm.d, (size_t)N * rowb, n_src * rowb, B,
                                hipMemcpyDeviceToDevice, st));
        HIPCHK(hipMemcpy2DAsync(s->tsrc, (size_t)n_src * 4, s->img + seq_of(p0), (size_t)NS * 4, (size_t)n_src * 4, B,
                                hipMemcpyDeviceToDevice, st));
        for (int j = 1; j <= o.K; ++j) {
          ssd_draft_head* h = (hor ? src.hh : src.vh)[j - 1];
          head_forward(h, h->work, B * n_src, s->hsrc, s->tsrc, st);
          const int dq = seq_of(p0 + j * step);  // a run or a row: contiguous in the sequence
          HIPCHK(hipMemcpy2DAsync(s->img + dq, (size_t)NS * 4, h->work.out, (size_t)n_src * 4, (size_t)n_src * 4, B,
                                  hipMemcpyDeviceToDevice, st));
          if (use_q)
            HIPCHK(hipMemcpy2DAsync(s->qtab + (size_t)dq * dm.Vimg, (size_t)NS * dm.Vimg * 4, h->work.logits,
                                    (size_t)n_src * dm.Vimg * 4, (size_t)n_src * dm.Vimg * 4, B,
                                    hipMemcpyDeviceToDevice, st));
        }
        continue;
      }
      if (o.kind == 1 && fuse[i]) {
        pending = &o;  // runs as the fixed prefix of the next verify pass
        continue;
      }
      // the pass's block: this op's, behind the pending commit's when there is one
      const int Kc = (o.kind == 0 && pending) ? pending->K : 0;
      const int start = o.start - Kc, K = o.K + Kc;
      HIPCHK(hipMemcpy2DAsync(s->tok, (size_t)K * 4, s->img + start, (size_t)NS * 4, (size_t)K * 4, B,
                              hipMemcpyDeviceToDevice, st));
      if (s->cfg)
        HIPCHK(hipMemcpyAsync(s->tok + (size_t)B * K, s->tok, (size_t)B * K * 4, hipMemcpyDeviceToDevice, st));
      if (o.kind == 0) {
        if (use_q) {
          // first round of a position: its reference is its draft distribution
          // (positions that already hold a reference keep it; a committed prefix's
          // are dropped by its commit below)
          set_ref_rows(B, K, NS, dm.Vimg, s->qtab + (size_t)start * dm.Vimg, s->d_f, s->ref, s->ref_flag, s->ring,
                       1, st);
        }
        run_forward(s, K, 0);
        if (s->cfg) cfg_mix(B, K, dm.Vimg, s->cfg_w, s->logits, s->carry, s->mlog, s->mcarry, st);
        const int rr = std::min(o.rib, NCNT_ROUNDS - 1);
        a.K = K;
        a.n_fixed = Kc + o.nf;  // the committed prefix is fixed
        a.round = (unsigned)o.rnd;
        a.count = s->cnt + (size_t)rr * Bs;
        select_tokens(a, st);
        HIPCHK(hipMemcpy2DAsync(s->img + start, (size_t)NS * 4, s->tok, (size_t)K * 4, (size_t)K * 4, B,
                                hipMemcpyDeviceToDevice, st));
        ++nv;
        int n_eol = 0;  // end-of-line slots are not verified
        for (int k = 0; eol && k < o.K; ++k) n_eol += (o.start + k) % RW == W;
        const int64_t np = (int64_t)B * (o.K - o.nf - n_eol);
        proposed += np;
        prop_round[rr] += np;
        if (Kc > 0) {  // the prefix's KV is final: commit it
          commit_prefix(Bs, K, Kc, dm.Vimg, s->logits, s->carry, s->d_f, s->ref_flag, s->ring, st);
          for (int b = 0; b < Bs; ++b) s->f[b] += Kc;
          keep_states(start, Kc, K);
          pending = nullptr;
        }
      } else {
        run_forward(s, o.K, 1);
        commit_update(Bs, -o.K, dm.Vimg, s->logits, s->carry, s->d_f, s->ref_flag, s->ring, st);
        for (int b = 0; b < Bs; ++b) s->f[b] += o.K;
        keep_states(o.start, o.K, o.K);
      }
      ++passes;
    }
    HIPCHK(hipGetLastError());
    // image positions only (rows of W out of rows of RW; the strict decode's slack left out)
    if (trunc)
      HIPCHK(hipMemcpy2DAsync(out_tokens, (size_t)N * 4, s->img, (size_t)NS * 4, (size_t)N * 4, B, hipMemcpyDefault,
                              st));
    else
      HIPCHK(hipMemcpy2DAsync(out_tokens, (size_t)W * 4, s->img, (size_t)RW * 4, (size_t)W * 4, (size_t)B * H,
                              hipMemcpyDefault, st));
    if (plant) HIPCHK(hipMemcpyAsync(src.table, s->ptab, (size_t)B * N * 4, hipMemcpyDefault, st));
    if (!trunc) HIPCHK(hipMemcpyAsync(hc.data(), s->cnt, hc.size() * 4, hipMemcpyDeviceToHost, st));
    fwd_abort_fetch(s);
    HIPCHK(hipStreamSynchronize(st));
    fwd_abort_check(s);
    m->prof.flush();
  } catch (HipError& e) {
    m->poisoned = true;
    return fail(SSD_E_DEVICE, "%s: %s", e.what, hipGetErrorString(e.e));
  }
  if (stats) {
    *stats = ssd_stats{};
    stats->passes = passes;
    stats->verify_rounds = nv;
    stats->proposed = proposed;
    if (trunc) {
      stats->accepted = acc_trunc;
      stats->accepted_round[0] = acc_trunc;
      stats->proposed_round[0] = proposed;
    } else {
      int64_t acc = 0;
      for (int r = 0; r < NCNT_ROUNDS; ++r) {
        int64_t ar = 0;
        for (int b = 0; b < B; ++b) ar += hc[(size_t)r * Bs + b];
        stats->accepted_round[r] = ar;
        stats->proposed_round[r] = prop_round[r];
        acc += ar;
      }
      stats->accepted = acc;
    }
    stats->wall_ns = (int64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                         std::chrono::steady_clock::now() - t_call).count();
  }
  return SSD_OK;
}

}  // namespace

ssd_status ssd_decode_image(ssd_model* m, const ssd_schedule* sc, int32_t B, int32_t P, const int32_t* prefix,
                            const int32_t* drafts, const float* draft_logits, int32_t* out_tokens, ssd_stats* stats,
                            void* stream) {
  g_err.clear();
  if (!m || !sc || !prefix || !drafts || !out_tokens) return fail(SSD_E_INVAL, "NULL argument");
  DraftSource src;
  src.drafts = drafts;
  src.draft_logits = draft_logits;
  return decode_impl(m, sc, B, P, prefix, src, out_tokens, stats, stream);
}

ssd_status ssd_plant_image(ssd_model* m, const ssd_schedule* sc, int32_t B, int32_t P, const int32_t* prefix,
                           const uint8_t* keep, const int32_t* repl, int32_t* drafts_out, int32_t* out_tokens,
                           ssd_stats* stats, void* stream) {
  g_err.clear();
  if (!m || !sc || !prefix || !keep || !repl || !drafts_out || !out_tokens) return fail(SSD_E_INVAL, "NULL argument");
  DraftSource src;
  src.keep = keep;
  src.repl = repl;
  src.table = drafts_out;
  return decode_impl(m, sc, B, P, prefix, src, out_tokens, stats, stream);
}

ssd_status ssd_decode_image_heads(ssd_model* m, const ssd_schedule* sc, int32_t B, int32_t P, const int32_t* prefix,
                                  ssd_draft_head* const* h_heads, int32_t n_h, ssd_draft_head* const* v_heads,
                                  int32_t n_v, int32_t* out_tokens, ssd_stats* stats, void* stream) {
  g_err.clear();
  if (!m || !sc || !prefix || !out_tokens) return fail(SSD_E_INVAL, "NULL argument");
  if (n_h < 0 || n_v < 0 || (n_h > 0 && !h_heads) || (n_v > 0 && !v_heads))
    return fail(SSD_E_INVAL, "bad head lists");
  static ssd_draft_head* const none[1] = {nullptr};
  DraftSource src;
  src.hh = n_h > 0 ? h_heads : none;
  src.nh = n_h;
  src.vh = n_v > 0 ? v_heads : none;
  src.nv = n_v;
  return decode_impl(m, sc, B, P, prefix, src, out_tokens, stats, stream);
}

}  // extern "C"
