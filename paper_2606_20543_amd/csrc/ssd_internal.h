// Internal declarations of the SSD verify-step library (gfx950).
//
// Data layout in HBM (all row-major unless stated):
//   residual x        fp32 [M][d]
//   xn                act [M][d]              g * x: the GEMM input after an RMSNorm
//   ssq               fp32 [parts][Mmax]      partial sums of x^2 per token (producer feature blocks)
//   q                 act [B][Hkv][rows_pad x D as 16x32 tiles]   bf16 models; query row
//                     r = head_in_group * K + k, rows_pad = K*g rounded up to 32
//                     (fp32 models: [B][Hq][K][D] row-major)
//   K cache           model dtype [L][B][Hkv][Lmax x D as 16x32 tiles]   (bf16; fp32: [Lmax][D])
//   V cache (transp.) model dtype [L][B][Hkv][D x Lmax as 16x32 tiles]   (bf16; fp32: [D][Lmax])
// A "16x32 tile" array stores each 16-row x 32-column tile (row-major tile
// order) as one MFMA operand: 64 lanes x 8 elements, 1 KiB in bf16, so a wave
// reads a whole tile with one coalesced 16-byte load per lane (tile16x32_index,
// vtile_index).
//   o                 act [M][Hq*D]           attention output
//   h                 act [M][d_ff]           SwiGLU product
//   logits            fp32 [M][V_img]
// "act" buffers of bf16 models are two bf16 planes, hi = bf16(v) and
// lo = bf16(v - hi), `plane` elements apart: an fp32 activation as a pair of
// MFMA operands (hi + lo carries v to 2^-17 relative).  fp32 models store
// fp32 in the first plane only.
// bf16 weight matrices W[N][K] are prepacked into 16x32 MFMA A-operand tiles:
//   tile (nb, kb) = 64 lanes x 8 bf16, lane l holds W[nb*16 + l%16][kb*32 + 8*(l/16) + e]
//   tiles ordered nb-major, so one wave reads 1 KiB contiguous per tile.
// Row permutations applied at packing so that each lane's four consecutive
// output features hold two (even, odd) pairs an epilogue needs together:
//   q/k rows: within a head, packed row 2j <- dim j, 2j+1 <- dim j + D/2 (rotary pair)
//   w1/w3:    packed row 2j <- gate row j, 2j+1 <- up row j (SwiGLU pair)
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/ssd.h"

namespace ssd {

struct Dims {
  int L, d, Hq, Hkv, D, dff, V, img_lo, img_hi, Vimg;
  bool bf16;
  float eps, theta;
};

enum EpiKind { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

// Arguments of a GEMM epilogue.  Token index t (0..M-1 of the whole call)
// maps to sequence b = t / Kblk and block position k = t % Kblk.
struct EpiArgs {
  int kind;
  int Kblk;
  const int* f;          // [B] block start positions (device)
  // rms scale: r_t = 1/sqrt(sum_p ssq[p*ssq_ld + t] / d + eps); ssq == nullptr -> r = 1
  const float* ssq;
  int ssq_parts, ssq_ld;
  int ssq_off, ssq_step;  // token t reads column ssq_off + t * ssq_step
  float inv_d, eps;
  // EPI_QKV
  void* q;
  void* kc;
  void* vc;
  int Lmax, Hq, Hkv, D;
  int qrows_pad;         // q_rows_pad(Kblk, Hq / Hkv): rows per KV head of the tiled q (bf16 models)
  const float2* rope;    // [Lmax][D/2] (cos, sin)
  // EPI_RESID: x += v; xn = bf16(gnext * x); ssq_out[fb][t] = sum over the block's features of x^2
  float* x;
  void* xn;
  const float* gnext;
  float* ssq_out;
  int ssq_out_ld;
  // EPI_SWIGLU
  void* h;
  // EPI_LOGITS
  float* logits;
  // common leading dimensions (elements)
  int ld;                // x / xn / h / logits row length
  // plane strides (elements) of the split activation buffers
  size_t q_plane, xn_plane, h_plane;
};

// Device model (owned by ssd_model)
struct LayerW {
  float* g1;
  float* g2;
  void* wqkv;  // N = (Hq + 2 Hkv) D, K = d   (packed)
  void* wo;    // N = d, K = Hq D
  void* w13;   // N = 2 dff, K = d
  void* w2;    // N = d, K = dff
};

// Element (row, col) of a [rows][cols] array stored as 16x32 operand tiles:
// lane = row%16 + 16*((col%32)/8) holds cols 8-aligned, element col%8 (the
// A/B operand layout of v_mfma_f32_16x16x32_bf16).
__host__ __device__ inline size_t tile16x32_index(int row, int col, int cols) {
  return ((size_t)(row >> 4) * (cols >> 5) + (col >> 5)) * 512 + (size_t)((((col & 31) >> 3) << 4) + (row & 15)) * 8 +
         (col & 7);
}
// Element (d, key) of the transposed V cache [D][Lmax] as 16x32 tiles of
// (16 dims x 32 keys), keys of a tile permuted so that lane d%16 + 16*g holds
// keys 4g..4g+3 and 16+4g..16+4g+3 (the A operand of O^T = V^T P^T whose
// P^T columns come straight from the S^T accumulators).
__host__ __device__ inline size_t vtile_index(int d, int key, int Lmax) {
  const int kk = key & 31;
  const int g = (kk & 15) >> 2, e = (kk & 3) + ((kk >> 4) << 2);
  return ((size_t)(d >> 4) * (Lmax >> 5) + (key >> 5)) * 512 + (size_t)(g * 16 + (d & 15)) * 8 + e;
}
// query rows per KV head padded for the tiled q layout
__host__ __device__ inline int q_rows_pad(int K, int g) { return ((K * g + 31) / 32) * 32; }

// Most partial sums of x^2 per token a GEMM's 1/rms prologue accepts (the
// producing GEMM writes one per 64-feature block: d_model <= 8192).
constexpr int GEMM_RMS_MAX_PARTS = 128;

// GEMM launch plan for one (M, N, K) problem.
struct GemmPlan {
  int MT, NT, KCB;  // token tiles, feature tiles per wave, 32-k blocks per chunk
  int WV;           // waves per workgroup (4, or 6..16 for one-burst wide workgroups)
  int S;            // K splits
  int n_fb;         // feature blocks
  int kchunks;      // chunks per split
  int bn;           // features per workgroup
  int xcd;          // >0: workgroups that reduce together share one XCD (n XCDs); 0: fenced reduction
  int tile;         // 1: tiled kernel for more than 64 rows (128-row tiles, K split only to fill the CUs);
                    // 3: 128 x 256 tiles of eight waves, both operands by LDS DMA
  int m_tiles;      // tiled: 128-row tiles
  int depth;        // tiled: register stages of the K pipeline (2 or 4)
  int tail_fb;      // tile 3, > 0: feature blocks [0, tail_fb) in one launch of whole tiles, the rest
  int tail_S;       //   in a second launch with K split tail_S ways (a last round that would run part empty)
  int tail_nt;      //   3: the rest as whole 128 x 192 tiles instead (tail_S 1), else 0
};
// split-K arrival counters a plan uses (tiled plans: one per output tile, when split)
inline int gemm_counters(const GemmPlan& p) {
  if (p.tile && p.tail_fb) return p.tail_nt ? 0 : (p.n_fb - p.tail_fb) * p.m_tiles;
  return p.tile ? (p.S > 1 ? p.n_fb * p.m_tiles : 0) : p.n_fb;
}
// Row counts that cover every plan class: up to 16, 32 and 64 rows, 65..128
// (one 128-row tile, or 64-row streaming tiles for shapes the tiled kernel
// does not take) and each count of 128-row tiles up to 256 (a split plan has
// fewer than 256 output tiles).  Sizing a workspace over these bounds every
// plan of any row count.
inline std::vector<int> gemm_row_classes() {
  std::vector<int> v = {1, 16, 17, 32, 33, 64, 65, 128};
  for (int t = 2; t <= 256; ++t) v.push_back(128 * t);
  return v;
}
// most per-row partial sums of x^2 a plan of output width N writes (one per
// feature block; no plan has blocks narrower than 64 features)
inline int gemm_max_parts(int N) { return (N + 63) / 64; }

// Cross-workgroup reductions (split-K partials, attention key chunks).  The
// workgroups of one reduction group are mapped onto one XCD, so their
// partials meet in that XCD's L2 and the last arrival needs no device-scope
// fence (no L2 write-back/invalidate).  Workgroup w runs on XCD w % X; group g
// lives on XCD g % X as its (g / X)-th group there.
__host__ __device__ inline int xcd_grid(int groups, int per_group, int X) {
  return X > 0 ? ((groups + X - 1) / X) * X * per_group : groups * per_group;
}
// -> (group, member) of workgroup w; group >= groups means idle
__host__ __device__ inline void xcd_unmap(int w, int per_group, int X, int& group, int& member) {
  if (X > 0) {
    const int x = w % X, slot = w / X;
    group = (slot / per_group) * X + x;
    member = slot % per_group;
  } else {
    group = w / per_group;
    member = w % per_group;
  }
}

// Workgroup barrier that orders LDS only: waits for this wave's LDS accesses,
// not for its outstanding global loads (a full __syncthreads() fence waits for
// every load in flight, which would stall a prefetched weight burst).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Measurement hook (host side).  While set, the GEMM and attention launchers
// start each kernel through hipExtLaunchKernelGGL with a start/stop event pair
// from the timer: the events take the dispatch's own begin/end timestamps, so
// no marker packet sits between consecutive kernels.  Per thread; set around
// one launch sequence.
struct LaunchTimer {
  virtual ~LaunchTimer() = default;
  virtual void next(hipEvent_t& start, hipEvent_t& stop) = 0;
};
extern thread_local LaunchTimer* g_launch_timer;

template <typename Kern, typename... Args>
inline void launch_timed(Kern kernel, dim3 grid, dim3 block, hipStream_t st, Args... args) {
  if (g_launch_timer) {
    hipEvent_t a, b;
    g_launch_timer->next(a, b);
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, a, b, 0, args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
  }
}

// ---- launchers (kernels_*.hip) ----
GemmPlan gemm_plan_bf16(int M, int N, int K, int xcd);
size_t gemm_partials_floats(const GemmPlan& p, int M);
// y = W x for split inputs in[M][K] (row stride ld_in, lo plane in_plane elements after hi); epilogue per `epi`.
void gemm_bf16(const GemmPlan& p, const void* Wpacked, int N, int K, const void* in, size_t in_plane, int ld_in,
               int M, const EpiArgs& epi, float* partials, unsigned* counters, hipStream_t st);
void gemm_f32(const float* W, int N, int K, const float* in, int ld_in, int M, const EpiArgs& epi, hipStream_t st);

void pack_bf16_tiles(const uint16_t* src, const int* rowmap, int N, int K, void* dst, hipStream_t st);
void gather_rows_f32(const float* src, const int* rowmap, int N, int K, float* dst, hipStream_t st);

// x[t] = E[tok[t]]; xn = g * x (split planes for bf16 models); ssq[t] = sum x^2 (one part)
void embed(const Dims& dm, const void* emb, const int* tok, int M, const float* g, float* x, void* xn,
           size_t xn_plane, float* ssq, hipStream_t st);
// fp32 path: xn = g * x, ssq[t] = sum x^2 (one part)
void norm_rows_f32(const float* x, int M, int d, const float* g, float* xn, float* ssq, hipStream_t st);

struct AttnKArgs {
  const uint16_t* q;   // [B][Hkv][qrows_pad x D tiles], hi plane then lo plane (q_plane elements apart)
  const uint16_t* kc;  // [B][Hkv][Lmax x D tiles]
  const uint16_t* vc;  // [B][Hkv][D x Lmax tiles, keys permuted]
  uint16_t* o;         // [B*K][Hq*D], hi plane then lo plane (o_plane elements apart)
  size_t q_plane, o_plane;
  float* opart;        // [groups][nchunk][QPW*16][D]   chunk partial O (relative to the chunk max)
  float2* spart;       // [groups][nchunk][QPW*16]      chunk (max, sum), log2 domain
  unsigned* counters;  // [groups]
  const int* f;
  int K, Hq, Hkv, g, Lmax, rows, qrows_pad, chunk, nchunk, nqg, groups, heads, xcd;
  float scale_log2;
};

// ---- persistent forward pass (kernels_fwd.hip) ----
enum FwdKind { FWD_GEMM = 0, FWD_ATTN = 1 };
// A GEMM phase: 64 output features x (bursts x 512) k per work item,
// items = xcd_grid(n_fb, S, xcd) (item -> (feature block, split) by xcd_unmap),
// S = K / (bursts x 512).
struct FwdGemm {
  const void* W;            // packed weights
  int N, K, KB, n_fb, S, bursts, items, M;
  const uint16_t* in;       // split input planes [M][ld_in]
  size_t in_plane;
  int ld_in;
  // K-slice s (features [s*512, (s+1)*512) of the input) needs producer units
  // [s*512*dep_scale/dep_width, ceil((s+1)*512*dep_scale/dep_width)) of `dep`
  // (dep_units > 0: every K-slice needs all units [0, dep_units) instead;
  // dep_att: the units are attention query groups, the slice needs those of
  // its heads' KV heads)
  const unsigned* dep;      // nullptr: input ready before launch
  int dep_width, dep_scale, dep_units, dep_att, dep_layer;
  // the epilogue's 1/rms needs all rms_units units of rms_dep
  const unsigned* rms_dep;
  int rms_units, rms_layer;
  float* part;
  unsigned* counters;
  unsigned* out_flags;      // one per feature block (nullptr: none)
  int out_layer;
  EpiArgs epi;
};
// An attention phase (geometry in FwdArgs::att; per-layer caches here).
struct FwdAttn {
  const unsigned* dep;      // QKV unit flags
  int dep_width, qN, kN, layer;
  const void* kc;
  const void* vc;
  unsigned* out_flags;      // one per query group
};
// Work item i of a phase runs on workgroup (i + rot) % grid (rot a multiple
// of the XCD count): consecutive phases start on different workgroups, so the
// workgroups still finishing one phase are not the first ones the next needs.
struct FwdPhase {
  int kind;
  int rot;
  FwdGemm g;
  FwdAttn a;
};
// Flag values are epoch_base + layer index + 1 (epoch_base = pass * (L + 1)).
struct FwdArgs {
  const FwdPhase* phases;   // device
  int n_phases;
  int xcd;
  unsigned* abort_flag;
  unsigned spin_limit;
  unsigned epoch_base;
  AttnKArgs att;            // attention geometry of this pass (caches per phase)
  int att_items;
  int* probe;               // non-null: workgroup w writes its XCD index to probe[w] first
};
hipError_t fwd_persistent(const FwdArgs& a, int MT, int D, int grid, hipStream_t st);
int fwd_max_grid(int MT, int D);  // co-resident workgroups of the persistent kernel (0: unsupported)

struct AttnPlan {
  int chunk;      // keys per workgroup
  int nchunk;     // chunks covering max context
  int qpw;        // query tiles per wave
  int qs = 0;     // 1: the waves split the query rows (query group = 4 * qpw tiles), else the keys
  int nqg;        // query groups
  int rows;       // query rows per (b, kv head) = K * g
  int xcd;        // see xcd_grid
  int group_rows() const { return (qs ? 4 : 1) * qpw * 16; }
};
// grid > 0: a plan for the persistent forward pass (one query tile per work
// item, items fitting `grid` workgroups where possible)
AttnPlan attn_plan(const Dims& dm, int B, int K, int max_ctx_now, int xcd, int grid = 0);
AttnKArgs attn_args(const Dims& dm, const AttnPlan& p, int B, int K, const int* f, const void* q, size_t q_plane,
                    const void* kc, const void* vc, int Lmax, void* o, size_t o_plane, float* partials,
                    unsigned* counters);
int attn_items(const AttnKArgs& a);  // work items (workgroups) of one attention call
size_t attn_partials_floats(const Dims& dm, const AttnPlan& p, int B);
void attention_bf16(const Dims& dm, const AttnPlan& p, int B, int K, const int* f, const void* q, size_t q_plane,
                    const void* kc, const void* vc, int Lmax, void* o, size_t o_plane, float* partials,
                    unsigned* counters, hipStream_t st);
void attention_f32(const Dims& dm, int B, int K, const int* f, const float* q, const float* kc, const float* vc,
                   int Lmax, float* o, hipStream_t st);

struct SelectArgs {
  int rule, top_k;
  double temperature;
  unsigned long long seed;
  unsigned round;
  int n_fixed, K, B, Vimg, img_lo;
  int truncate;
  const int* f;
  int* tokens;             // [B][K] absolute ids (in/out)
  const float* logits;     // [B*K][Vimg]
  const float* carry;      // [B][Vimg]
  float* ref;              // ring [B][ring][Vimg]
  int* ref_flag;           // ring [B][ring]
  int ring;
  unsigned char* accept;   // [B][K]
  int* count;              // [B]
  int* amax;               // [B][K] greedy argmax (truncate mode)
  int eol_period = 0;      // > 0: sequence position p is a fixed end-of-line token
  int eol_base = 0;        //   when (p - eol_base) % eol_period == eol_period - 1
};
void select_tokens(const SelectArgs& a, hipStream_t st);
// truncate mode: leading accepted run, f update, pending token
void truncate_finalize(const SelectArgs& a, int* f, hipStream_t st);
// commit bookkeeping: carry <- logits[b*K + K-1]; f += K; clear ring flags of committed positions
void commit_update(int B, int K, int Vimg, const float* logits, float* carry, int* f, int* ref_flag, int ring,
                   hipStream_t st);
// commit of the first Kc rows of a pass of rps rows per sequence (the rest a
// verify block): carry <- logits row Kc-1, f += Kc, ring flags of the committed
// positions cleared
void commit_prefix(int B, int rps, int Kc, int Vimg, const float* logits, float* carry, int* f, int* ref_flag,
                   int ring, hipStream_t st);
// greedy argmax of a logits row placed at image index f[b] - P + pos_off: a
// planted draft (keep/repl given) or the token itself (keep == nullptr)
struct PlaceArgs {
  const float* logits;        // row of sequence b at logits + b * row_stride
  size_t row_stride;
  int Vimg, img_lo;
  const int* f;               // [B] frontier (sequence positions)
  int P, pos_off, x_end;      // image index x = f[b] - P + pos_off, valid in [0, x_end)
  int* img;                   // working grid, row b at img + b * img_stride (absolute ids)
  size_t img_stride;
  const unsigned char* keep;  // [B][x_end] or nullptr
  const int* repl;            // [B][x_end] codes in [0, Vimg - 1)
  int* table;                 // [B][x_end] planted drafts out (absolute ids) or nullptr
  int* next_tok;              // [B] token of the next single-position pass or nullptr
  int* active;                // [B] gate or nullptr
};
void place_argmax(const PlaceArgs& a, int B, hipStream_t st);
// tok[b][k] = img[b][f[b] - P + k]
void gather_block(const int* img, int img_stride, const int* f, int P, int K, int B, int* tok, hipStream_t st);
// p[i] += delta
void add_i32(int* p, int n, int delta, hipStream_t st);
// fill helpers (graph-capture safe)
void fill_u32(unsigned* p, size_t n, unsigned v, hipStream_t st);
// out[w] = XCD index workgroup w ran on
void xcc_probe(int* out, int n_wg, hipStream_t st);
// references of block positions f+k <- src rows (b * rows_per_b + k); only_new keeps existing references
void set_ref_rows(int B, int K, int rows_per_b, int Vimg, const float* src, const int* f, float* ref, int* ref_flag,
                  int ring, int only_new, hipStream_t st);
// z = [h; e] split planes [R][2d] (plane elements apart) for a draft head
void draft_input_f32(const float* h, const float* emb, const int* tok, int R, int d, float* z, hipStream_t st);
void draft_input(const float* h, const void* emb, const int* tok, int R, int d, void* z, size_t plane,
                 hipStream_t st);
// guided logits l_u + w (l_c - l_u): rows [Bi][K] from the pass's [2*Bi][K] logits
// (K may be 0) and the carry [Bi] from [2*Bi]
void cfg_mix(int Bi, int K, int Vimg, float w, const float* logits, const float* carry, float* out_logits,
             float* out_carry, hipStream_t st);
void first_token(int B, int Vimg, int img_lo, const float* carry, int rule, int top_k, double temperature,
                 unsigned long long seed, const int* f, int* out_abs, int out_stride, hipStream_t st);

}  // namespace ssd
