// Host-side logic of libssd under AddressSanitizer and UndefinedBehaviorSanitizer,
// on the CPU (no GPU is touched): configuration validation and packed sizes,
// argument checks of every entry point, GEMM launch plans and their workspace
// sizes, the image pass plans, and the session workspace sizing.  Built with
// the library's host source included into this translation unit, so the
// internal (file-local) functions are callable; device code is not compiled.
#include "../../paper_2606_20543_amd/csrc/ssd_api.cpp"

#include <cstdio>

namespace {

int g_fail = 0;
#define CHECK(c)                                                         \
  do {                                                                   \
    if (!(c)) {                                                          \
      std::fprintf(stderr, "CHECK failed at line %d: %s\n", __LINE__, #c); \
      ++g_fail;                                                          \
    }                                                                    \
  } while (0)

ssd_model_config cfg_of(int L, int d, int Hq, int Hkv, int D, int f, int V, int lo, int hi, int dtype) {
  ssd_model_config c{};
  c.n_layers = L;
  c.d_model = d;
  c.n_heads = Hq;
  c.n_kv_heads = Hkv;
  c.head_dim = D;
  c.d_ff = f;
  c.vocab = V;
  c.img_lo = lo;
  c.img_hi = hi;
  c.dtype = dtype;
  c.rms_eps = 1e-5f;
  c.rope_theta = 1e4f;
  return c;
}

Dims dims_of(const ssd_model_config& c) {
  Dims dm{};
  dm.L = c.n_layers;
  dm.d = c.d_model;
  dm.Hq = c.n_heads;
  dm.Hkv = c.n_kv_heads;
  dm.D = c.head_dim;
  dm.dff = c.d_ff;
  dm.V = c.vocab;
  dm.img_lo = c.img_lo;
  dm.img_hi = c.img_hi;
  dm.Vimg = c.img_hi - c.img_lo;
  dm.bf16 = c.dtype == SSD_BF16;
  dm.eps = c.rms_eps;
  dm.theta = c.rope_theta;
  return dm;
}

}  // namespace

int main() {
  const ssd_model_config shapes[] = {
      cfg_of(2, 256, 4, 4, 64, 688, 1024, 0, 1024, SSD_F32),                  // tiny fp32
      cfg_of(24, 2048, 16, 16, 128, 5632, 16384, 0, 16384, SSD_BF16),         // 1B
      cfg_of(32, 4096, 32, 32, 128, 11008, 65536, 57344, 65536, SSD_BF16),    // 7B
      cfg_of(32, 4096, 32, 8, 128, 14336, 65536, 32768, 65536, SSD_BF16),     // 8B GQA
  };
  // 1. configurations: valid ones have a packed size, broken ones are refused
  for (const auto& c : shapes) {
    CHECK(ssd_weights_numel(&c) > 0);
    ssd_model_config b = c;
    b.n_kv_heads = 5;
    CHECK(ssd_weights_numel(&b) == -1);
    b = c;
    b.img_hi = c.vocab + 1;
    CHECK(ssd_weights_numel(&b) == -1);
    b = c;
    b.head_dim = 3;
    CHECK(ssd_weights_numel(&b) == -1);
    b = c;
    b.n_layers = 0;
    CHECK(ssd_weights_numel(&b) == -1);
  }
  CHECK(ssd_weights_numel(nullptr) == -1);
  // 2. argument checks before any device work
  ssd_model* mo = nullptr;
  ssd_session* so = nullptr;
  CHECK(ssd_init_model(nullptr, nullptr, nullptr, &mo) == SSD_E_INVAL);
  CHECK(ssd_init_model(&shapes[0], nullptr, nullptr, &mo) == SSD_E_INVAL);
  CHECK(ssd_prefill(nullptr, 1, 1, nullptr, 2, 1, nullptr, &so) == SSD_E_INVAL);
  ssd_verify_params vp{};
  CHECK(ssd_verify_step(nullptr, 1, nullptr, nullptr, &vp, nullptr, nullptr, nullptr, nullptr, nullptr) ==
        SSD_E_INVAL);
  ssd_schedule sc{};
  ssd_stats stv{};
  CHECK(ssd_decode_image(nullptr, &sc, 1, 1, nullptr, nullptr, nullptr, nullptr, &stv, nullptr) == SSD_E_INVAL);
  CHECK(ssd_plant_image(nullptr, &sc, 1, 1, nullptr, nullptr, nullptr, nullptr, nullptr, &stv, nullptr) ==
        SSD_E_INVAL);
  CHECK(ssd_decode_image_heads(nullptr, &sc, 1, 1, nullptr, nullptr, 0, nullptr, 0, nullptr, &stv, nullptr) ==
        SSD_E_INVAL);
  CHECK(ssd_draft_head_run(nullptr, 1, nullptr, nullptr, nullptr, nullptr) == SSD_E_INVAL);
  CHECK(ssd_draft_head_run_noalloc(nullptr, 1, nullptr, nullptr, nullptr, nullptr) == SSD_E_INVAL);
  CHECK(ssd_get_carry(nullptr, nullptr) == SSD_E_INVAL);
  CHECK(ssd_session_set_cfg(nullptr, 1.f) == SSD_E_INVAL);
  CHECK(ssd_profile(nullptr, 1) == SSD_E_INVAL);
  CHECK(ssd_profile_read(nullptr, nullptr, nullptr, nullptr, nullptr, 0) == SSD_E_INVAL);
  CHECK(std::strlen(ssd_last_error()) > 0);
  ssd_free_session(nullptr);
  ssd_free_model(nullptr);
  ssd_free_draft_head(nullptr);
  // 3. GEMM plans: exact tiling and workspace sizes for every projection shape
  for (const auto& c : shapes) {
    if (c.dtype != SSD_BF16) continue;
    const int d = c.d_model, D = c.head_dim, Nqkv = (c.n_heads + 2 * c.n_kv_heads) * D;
    const std::pair<int, int> nks[] = {{Nqkv, d}, {d, c.n_heads * D}, {2 * c.d_ff, d}, {d, c.d_ff},
                                       {c.img_hi - c.img_lo, d}, {d, 2 * d}, {4 * d, d}, {d, 2 * d}};
    for (const auto& nk : nks) {
      for (int M = 1; M <= 4352; M += (M < 160 ? 1 : 37)) {
        for (int X : {0, 8}) {
          GemmPlan p = gemm_plan_bf16(M, nk.first, nk.second, X);
          CHECK(p.n_fb * p.bn == nk.first);
          CHECK(p.S >= 1);
          CHECK(gemm_partials_floats(p, M) < ((size_t)1 << 40));
          CHECK(gemm_counters(p) >= 0);
        }
      }
    }
  }
  // 4. pass plans: the printed formula (k_h = 5, h_rounds = 1) for joint and staged groups
  for (int H : {1, 2, 5, 24, 64}) {
    for (int W : {1, 3, 24, 64}) {
      for (int kv : {1, 2, 3}) {
        for (int b : {0, 2, 5}) {
          for (int i : {0, 1}) {
            std::vector<Op> ops = make_plan(H, W, 5, 1, kv, b, i, false);
            long passes = 1;
            for (const Op& o : ops) passes += o.kind <= 1;
            long want = 1 + 2 * ((W - 1 + 4) / 5) + (W == 1 ? 1 : 0);
            for (int y = 1; y < H; y += kv) {
              const int m = std::min(kv, H - y);
              want += b + i * (m - 1) + m;
            }
            CHECK(passes == want);
            for (const Op& o : ops) CHECK(o.kind < 2 || o.K >= 1);
          }
        }
      }
    }
  }
  // 5. session workspace sizing (no persistent pass): finite and growing with the session
  for (const auto& c : shapes) {
    ssd_model m{};
    m.dm = dims_of(c);
    m.xcd = 8;
    size_t gp = 0, gc = 0, ap = 0, ac = 0, gp2 = 0, gc2 = 0, ap2 = 0, ac2 = 0;
    int parts = 0, parts2 = 0;
    size_workspaces(m.dm, &m, 1, 16, 8, 128, gp, gc, ap, ac, parts);
    size_workspaces(m.dm, &m, 8, 256, 128, 4416, gp2, gc2, ap2, ac2, parts2);
    CHECK(gp2 >= gp && gc2 >= gc && ap2 >= ap && ac2 >= ac && parts2 >= parts);
    CHECK(parts >= 1);
  }
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("host checks passed\n");
  return 0;
}
