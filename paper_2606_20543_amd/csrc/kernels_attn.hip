// Block-causal multi-query attention of the verify pass over the KV cache.
//
// A block of K tokens at positions [f, f+K) attends under the backbone's
// ordinary causal mask over raster positions: block token k (position f+k)
// sees cache slots [0, f+k].  The paper's backbone is used unmodified
// (Sec. 3.3), so no other mask exists; the drafted block simply occupies the
// next raster positions.
//
// bf16 path: a workgroup of four waves owns one key chunk of one query group
// (16 or 32 query rows of one sequence x KV head; the K*g rows of a KV head,
// g = query heads per KV head, are tiled by 16).  Wave w streams the chunk's
// 32-key blocks w, w+4, ..., with the next block's K and V tiles in flight
// while the current one is multiplied.  S^T = K Q^T and O^T = V^T P^T run on
// v_mfma_f32_16x16x32_bf16 with queries as the MFMA columns, so the softmax
// statistics of a query live in one lane column and need two cross-lane
// shuffles; the P^T operand is built in registers straight from the S^T
// accumulators (its key order is matched by reading the transposed V cache),
// so P never touches LDS.  The four waves' (max, sum, O) triples are merged
// through LDS.  A context is split into several chunks only when the chunks'
// shorter streams outweigh the cost of merging them (few query groups, long
// contexts) or to fill the chip (many query groups); chunks of one query group
// run on workgroups of one XCD, and the last to arrive combines them in chunk
// order.
#include "ssd_internal.h"

namespace ssd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint16_t f2bf_a(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

constexpr int AT_KEYS = 32;        // keys per wave step
constexpr int AT_STEP = 128;       // chunk granularity in keys (one workgroup step)
constexpr int AT_MAX_CHUNKS = 64;
// four waves per workgroup: one wave per SIMD, so a wave holds two K/V blocks
// (the one in use and the next) beside its queries and accumulators
template <int QPW>
struct AtShape {
  static constexpr int WAVES = 4;
  static constexpr int THREADS = WAVES * 64;
  static constexpr int STEP = WAVES * AT_KEYS;
};

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

// hi/lo bf16 planes of four consecutive fp32 values
__device__ __forceinline__ void store_split4(uint16_t* p, size_t plane, floatx4 v) {
  uint16_t hi[4], lo[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    hi[e] = f2bf_a(v[e]);
    lo[e] = f2bf_a(v[e] - __uint_as_float((uint32_t)hi[e] << 16));
  }
  uint2 w, x;
  w.x = (uint32_t)hi[0] | ((uint32_t)hi[1] << 16);
  w.y = (uint32_t)hi[2] | ((uint32_t)hi[3] << 16);
  x.x = (uint32_t)lo[0] | ((uint32_t)lo[1] << 16);
  x.y = (uint32_t)lo[2] | ((uint32_t)lo[3] << 16);
  *(uint2*)p = w;
  *(uint2*)(p + plane) = x;
}

// K and V operands of one 32-key block: K tiles (keys key0 + kt*16 + [0,16),
// dims kd*32 + [0,32)) are the A operands of S^T, V^T tiles (dims dt*16 + [0,16),
// keys key0 + [0,32)) those of O^T.  In the tiled caches each is 1 KiB
// contiguous in lane order: one coalesced 16-byte load per lane.  A block past
// the cache (a prefetch beyond the chunk) reloads the cache's last block.
template <int D>
struct KVTile {
  u32x4 k[2][D / 32];
  u32x4 v[D / 16];
};

template <int D>
__device__ __forceinline__ void load_kv(KVTile<D>& t, const uint16_t* kbase, const uint16_t* vbase, int key0,
                                        int Lmax, int lane) {
  const int kb = key0 < Lmax - 32 ? key0 : Lmax - 32;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int kd = 0; kd < D / 32; ++kd)
      t.k[kt][kd] = *(const u32x4*)(kbase + ((size_t)((kb >> 4) + kt) * (D / 32) + kd) * 512 + lane * 8);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt)
    t.v[dt] = *(const u32x4*)(vbase + ((size_t)dt * (Lmax >> 5) + (kb >> 5)) * 512 + lane * 8);
}

// one 32-key block through the online softmax of the wave's query tiles
template <int D, int QPW>
__device__ __forceinline__ void attend_block(const KVTile<D>& t, int key0, const bf16x8 (&qh)[QPW][D / 32],
                                             const bf16x8 (&ql)[QPW][D / 32], const int (&qpos)[QPW],
                                             float scale_log2, int grp, float (&m)[QPW], float (&l)[QPW],
                                             floatx4 (&O)[QPW][D / 16]) {
  constexpr int KD = D / 32, DT = D / 16;
  floatx4 s[2][QPW];
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int qt = 0; qt < QPW; ++qt) {
      floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kd = 0; kd < KD; ++kd) {
        const bf16x8 kf = __builtin_bit_cast(bf16x8, t.k[kt][kd]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qh[qt][kd], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, ql[qt][kd], acc, 0, 0, 0);
      }
      s[kt][qt] = acc;
    }
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    float sv[8];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = key0 + kt * 16 + 4 * grp + e;
        float v = s[kt][qt][e] * scale_log2;
        v = (key <= qpos[qt]) ? v : -INFINITY;
        sv[kt * 4 + e] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m[qt], mx);
    const bool none = (mnew == -INFINITY);
    const float alpha = none ? 1.f : exp2f(m[qt] - mnew);
    float ps = 0.f;
    uint16_t pb[8], pl[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float p = none ? 0.f : exp2f(sv[i] - mnew);
      ps += p;
      pb[i] = f2bf_a(p);
      pl[i] = f2bf_a(p - __uint_as_float((uint32_t)pb[i] << 16));
    }
    l[qt] = l[qt] * alpha + ps;
    m[qt] = mnew;
    const u32x4 pv = {(uint32_t)pb[0] | ((uint32_t)pb[1] << 16), (uint32_t)pb[2] | ((uint32_t)pb[3] << 16),
                      (uint32_t)pb[4] | ((uint32_t)pb[5] << 16), (uint32_t)pb[6] | ((uint32_t)pb[7] << 16)};
    const u32x4 pw = {(uint32_t)pl[0] | ((uint32_t)pl[1] << 16), (uint32_t)pl[2] | ((uint32_t)pl[3] << 16),
                      (uint32_t)pl[4] | ((uint32_t)pl[5] << 16), (uint32_t)pl[6] | ((uint32_t)pl[7] << 16)};
    const bf16x8 pf = __builtin_bit_cast(bf16x8, pv);
    const bf16x8 pg = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      O[qt][dt] *= alpha;
      const bf16x8 vf = __builtin_bit_cast(bf16x8, t.v[dt]);
      O[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, O[qt][dt], 0, 0, 0);
      O[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pg, O[qt][dt], 0, 0, 0);
    }
  }
}

// PF = 1: the next block's K/V tiles are loaded while the current one is used
template <int D, int QPW, int PF>
// one wave per SIMD: the register file holds two K/V blocks, the queries and
// the accumulators without the compiler sinking the prefetch loads
__global__ __launch_bounds__(AtShape<QPW>::THREADS) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attn_bf16_kernel(AttnKArgs a) {
  constexpr int NW = AtShape<QPW>::WAVES, NTH = AtShape<QPW>::THREADS, STEP = AtShape<QPW>::STEP;
  constexpr int KD = D / 32;   // 32-wide k steps over the head dimension
  constexpr int DT = D / 16;   // 16-row d tiles of O^T
  constexpr int ROWS = QPW * 16;
  constexpr int RS = D + 4;    // LDS row stride (floats): rows of one wave fall on different banks
  constexpr int NOUT = ROWS * D / 4;                          // float4 outputs of the workgroup
  constexpr int NV = (NOUT + NTH - 1) / NTH;    // per thread
  static_assert(2 * AT_MAX_CHUNKS * ROWS <= NW * ROWS * RS, "chunk statistics fit the O stage");
  __shared__ __align__(16) float sm_o[NW * ROWS * RS];
  __shared__ float sm_m[NW * ROWS], sm_l[NW * ROWS];
  __shared__ int is_last;

  // single chunk: the query groups of one (sequence, KV head) share an XCD
  // (they read the same K/V); several chunks: the chunks of one query group
  // share an XCD (their partials meet in its L2)
  int grp_id, c, z, qg;
  if (a.nchunk == 1) {
    xcd_unmap(blockIdx.x, a.nqg, a.xcd, z, qg);
    if (z >= a.heads) return;
    grp_id = z * a.nqg + qg;
    c = 0;
  } else {
    xcd_unmap(blockIdx.x, a.nchunk, a.xcd, grp_id, c);
    if (grp_id >= a.groups) return;
    qg = grp_id % a.nqg;
    z = grp_id / a.nqg;
  }
  const int b = z / a.Hkv, hkv = z - b * a.Hkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int fb = a.f[b];
  const int ctx = fb + a.K;
  const int nch = (ctx + a.chunk - 1) / a.chunk;
  if (c >= nch) return;  // whole workgroup, before any barrier
  const int kbeg = c * a.chunk;
  const int kend = min(kbeg + a.chunk, ctx);
  const int rbase = qg * ROWS;

  const uint16_t* kbase = a.kc + ((size_t)b * a.Hkv + hkv) * a.Lmax * D;
  const uint16_t* vbase = a.vc + ((size_t)b * a.Hkv + hkv) * (size_t)D * a.Lmax;
  const int first = kbeg + wave * AT_KEYS;
  const int nit = first < kend ? (kend - first + STEP - 1) / STEP : 0;

  // first K/V block in flight together with the queries.  K/V loads are never
  // conditional (a branch around loads makes the compiler wait for all of them
  // at the join): rows past the cache are clamped, and a block past the chunk
  // is loaded but never used.
  KVTile<D> ta, tb;
  load_kv<D>(ta, kbase, vbase, first, a.Lmax, lane);

  // query fragments (B operand of S^T = K Q^T): lane holds row col of tile qt, d = 8*grp.. (+32 kd);
  // q is fp32 carried as hi + lo bf16 operands
  bf16x8 qh[QPW][KD], ql[QPW][KD];
  int qpos[QPW];
  const uint16_t* qbase = a.q + (size_t)z * a.qrows_pad * D;
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    const int r = rbase + qt * 16 + col;  // padded rows (r >= rows) exist and are masked
    qpos[qt] = r < a.rows ? fb + r % a.K : -1;
    const uint16_t* qp = qbase + ((size_t)((rbase >> 4) + qt) * KD) * 512 + lane * 8;
#pragma unroll
    for (int kd = 0; kd < KD; ++kd) {
      qh[qt][kd] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + kd * 512));
      ql[qt][kd] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + a.q_plane + kd * 512));
    }
  }

  float m[QPW], l[QPW];
  floatx4 O[QPW][DT];
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    m[qt] = -INFINITY;
    l[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) O[qt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  if constexpr (PF) {
    // the next block is loaded before the current one is used and taken over
    // at the end of every iteration (an unconditional use: the compiler can
    // neither sink the loads past a loop exit nor drop the overlap)
    for (int it = 0; it < nit; ++it) {
      const int key0 = first + it * STEP;
      load_kv<D>(tb, kbase, vbase, key0 + STEP, a.Lmax, lane);
      attend_block<D, QPW>(ta, key0, qh, ql, qpos, a.scale_log2, grp, m, l, O);
      ta = tb;
    }
  } else {
    for (int it = 0; it < nit; ++it) {
      const int key0 = first + it * STEP;
      attend_block<D, QPW>(ta, key0, qh, ql, qpos, a.scale_log2, grp, m, l, O);
      load_kv<D>(ta, kbase, vbase, key0 + STEP, a.Lmax, lane);
    }
  }

  // stage this wave's triple: O^T accumulator element e of tile (qt, dt) is row
  // qt*16 + col, dims dt*16 + 4*grp + e
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    l[qt] += __shfl_xor(l[qt], 16);
    l[qt] += __shfl_xor(l[qt], 32);
    float* row = sm_o + (size_t)(wave * ROWS + qt * 16 + col) * RS;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *(floatx4*)(row + dt * 16 + 4 * grp) = O[qt][dt];
    if (grp == 0) {
      sm_m[wave * ROWS + qt * 16 + col] = m[qt];
      sm_l[wave * ROWS + qt * 16 + col] = l[qt];
    }
  }
  __syncthreads();

  // merge the waves: thread owns float4 slots idx = tid + NTH * i (row r, dims 4*d4..)
  floatx4 acc[NV];
  float Lr[NV], Mr[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int idx = threadIdx.x + NTH * i;
    const int ic = idx < NOUT ? idx : NOUT - 1;
    const int r = ic / (D / 4), d4 = ic - r * (D / 4);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, sm_m[w * ROWS + r]);
    float L = 0.f;
    floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = sm_m[w * ROWS + r];
      const float ew = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
      L += sm_l[w * ROWS + r] * ew;
      v += *(const floatx4*)(sm_o + (size_t)(w * ROWS + r) * RS + 4 * d4) * ew;
    }
    acc[i] = v;
    Lr[i] = L;
    Mr[i] = M;
  }

  if (nch == 1) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + NTH * i;
      if (idx >= NOUT) continue;
      const int r = idx / (D / 4), d4 = idx - r * (D / 4);
      const int rg = rbase + r;
      if (rg >= a.rows) continue;
      const int j = rg / a.K, k = rg - j * a.K;
      uint16_t* op = a.o + ((size_t)b * a.K + k) * (a.Hq * D) + (hkv * a.g + j) * D + 4 * d4;
      store_split4(op, a.o_plane, acc[i] * (1.f / Lr[i]));
    }
    return;
  }

  // publish the chunk's triple
  const size_t gbase = (size_t)grp_id * a.nchunk;
  {
    floatx4* Op = (floatx4*)(a.opart + (gbase + c) * ROWS * D);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + NTH * i;
      if (idx >= NOUT) continue;
      Op[idx] = acc[i];
      const int r = idx / (D / 4), d4 = idx - r * (D / 4);
      if (d4 == 0) a.spart[(gbase + c) * ROWS + r] = make_float2(Mr[i], Lr[i]);
    }
  }
  // partial stores acknowledged by this XCD's L2, then count the arrival
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (!a.xcd) __threadfence();  // chunks on different XCDs: write back through L2
    unsigned prev = atomicAdd(&a.counters[grp_id], 1u);
    is_last = (prev == (unsigned)(nch - 1));
    if (is_last && !a.xcd) __threadfence();
  }
  __syncthreads();
  if (!is_last) return;

  // last chunk: statistics of every (chunk, row) into LDS (parallel loads)
  float* cm = sm_o;                           // [nch][ROWS] chunk max
  float* cl = sm_o + AT_MAX_CHUNKS * ROWS;    // [nch][ROWS] chunk sum, then weight
  for (int i = threadIdx.x; i < nch * ROWS; i += NTH) {
    const float2 st = a.spart[gbase * ROWS + i];
    cm[i] = st.x;
    cl[i] = st.y;
  }
  __syncthreads();
  if (threadIdx.x < ROWS) {
    const int r = threadIdx.x;
    float M = -INFINITY;
    for (int cc = 0; cc < nch; ++cc) M = fmaxf(M, cm[cc * ROWS + r]);
    float L = 0.f;
    for (int cc = 0; cc < nch; ++cc) {
      const float lc = cl[cc * ROWS + r];
      const float w = (lc > 0.f) ? exp2f(cm[cc * ROWS + r] - M) : 0.f;
      L += lc * w;
      cl[cc * ROWS + r] = w;
    }
    sm_l[r] = L;
  }
  __syncthreads();
  // weighted sum of the chunk partials in chunk order; the slots' loads of
  // four chunks are in flight together
  const floatx4* G = (const floatx4*)(a.opart + gbase * ROWS * D);
  floatx4 v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int cc = 0; cc < nch; ++cc) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + NTH * i;
      const int ic = idx < NOUT ? idx : NOUT - 1;
      v[i] += G[(size_t)cc * NOUT + ic] * cl[cc * ROWS + ic / (D / 4)];
    }
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int idx = threadIdx.x + NTH * i;
    if (idx >= NOUT) continue;
    const int r = idx / (D / 4), d4 = idx - r * (D / 4);
    const int rg = rbase + r;
    if (rg >= a.rows) continue;
    const int j = rg / a.K, k = rg - j * a.K;
    uint16_t* op = a.o + ((size_t)b * a.K + k) * (a.Hq * D) + (hkv * a.g + j) * D + 4 * d4;
    store_split4(op, a.o_plane, v[i] * (1.f / sm_l[r]));
  }
  if (threadIdx.x == 0) a.counters[grp_id] = 0u;
}

AttnPlan attn_plan(const Dims& dm, int B, int K, int max_ctx_now, int xcd) {
  AttnPlan p;
  p.xcd = xcd;
  const int g = dm.Hq / dm.Hkv;
  p.rows = K * g;
  const int qt = (p.rows + 15) / 16;
  p.qpw = qt >= 4 ? 2 : 1;
  p.nqg = (qt + p.qpw - 1) / p.qpw;
  const long units = (long)B * dm.Hkv * p.nqg;
  const int ctx = max_ctx_now < 1 ? 1 : max_ctx_now;
  auto chunk_for = [&](int n) {  // whole workgroup steps covering ctx in n chunks
    const int per = (ctx + n - 1) / n;
    return ((per + AT_STEP - 1) / AT_STEP) * AT_STEP;
  };
  int best = 1;
  if (units >= 256) {
    // many query groups: the chip is full, chunks only bound the per-workgroup stream
    int chunk = AT_STEP;
    while ((chunk < 16 * AT_STEP && units * ((ctx + chunk - 1) / chunk) > 1024) ||
           (ctx + chunk - 1) / chunk > AT_MAX_CHUNKS)
      chunk *= 2;
    p.chunk = chunk;
  } else {
    // few query groups: a chunk costs about 0.85 us per 128-key step of its
    // workgroup, a split adds the partial publish and the merge (about
    // 1.6 us + 0.08 us per chunk); measured on MI355X with D = 128
    double best_t = 1e30;
    for (int n = 1; n <= AT_MAX_CHUNKS && units * n <= 256; ++n) {
      const int ch = chunk_for(n);
      const int nn = (ctx + ch - 1) / ch;
      if (nn != n) continue;
      const double t = 0.85 * (ch / AT_STEP) * (dm.D / 128.0) + (n > 1 ? 1.6 + 0.08 * n : 0.0);
      if (t < best_t - 1e-9) {
        best_t = t;
        best = n;
      }
    }
    p.chunk = chunk_for(best);
  }
  p.nchunk = (ctx + p.chunk - 1) / p.chunk;
  return p;
}

size_t attn_partials_floats(const Dims& dm, const AttnPlan& p, int B) {
  return (size_t)B * dm.Hkv * p.nqg * p.nchunk * p.qpw * 16 * (dm.D + 2);
}

template <int D, int QPW>
static void launch_attn(const AttnKArgs& a, hipStream_t st) {
  const int grid = a.nchunk == 1 ? xcd_grid(a.heads, a.nqg, a.xcd) : xcd_grid(a.groups, a.nchunk, a.xcd);
  launch_timed(attn_bf16_kernel<D, QPW, 1>, dim3(grid), dim3(AtShape<QPW>::THREADS), st, a);
}

void attention_bf16(const Dims& dm, const AttnPlan& p, int B, int K, const int* f, const void* q, size_t q_plane,
                    const void* kc, const void* vc, int Lmax, void* o, size_t o_plane, float* partials,
                    unsigned* counters, hipStream_t st) {
  AttnKArgs a;
  a.q = (const uint16_t*)q;
  a.kc = (const uint16_t*)kc;
  a.vc = (const uint16_t*)vc;
  a.o = (uint16_t*)o;
  a.q_plane = q_plane;
  a.o_plane = o_plane;
  a.heads = B * dm.Hkv;
  a.groups = a.heads * p.nqg;
  // partial O block first, then the (max, sum) pairs (offset is a multiple of D floats: 8-byte aligned)
  a.opart = partials;
  a.spart = (float2*)(partials + (size_t)a.groups * p.nchunk * p.qpw * 16 * dm.D);
  a.counters = counters;
  a.f = f;
  a.K = K;
  a.Hq = dm.Hq;
  a.Hkv = dm.Hkv;
  a.g = dm.Hq / dm.Hkv;
  a.Lmax = Lmax;
  a.rows = p.rows;
  a.qrows_pad = q_rows_pad(K, a.g);
  a.chunk = p.chunk;
  a.nchunk = p.nchunk;
  a.nqg = p.nqg;
  a.xcd = p.xcd;
  a.scale_log2 = 1.4426950408889634f / sqrtf((float)dm.D);
  if (dm.D == 128) {
    if (p.qpw == 2) launch_attn<128, 2>(a, st);
    else launch_attn<128, 1>(a, st);
  } else {
    if (p.qpw == 2) launch_attn<64, 2>(a, st);
    else launch_attn<64, 1>(a, st);
  }
}

// ---------------- fp32 path ----------------
// One workgroup per (query, head, sequence): scores in LDS, two-pass softmax.
constexpr int F32_MAX_CTX = 4096;

__global__ __launch_bounds__(256) void attn_f32_kernel(int K, int Hq, int Hkv, int D, int Lmax, const int* f,
                                                       const float* q, const float* kc, const float* vc, float* o,
                                                       float scale) {
  __shared__ float sc[F32_MAX_CTX];
  __shared__ float red[256];
  const int k = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int g = Hq / Hkv, hkv = h / g;
  const int pos = f[b] + k;
  const int n = pos + 1;
  const float* qp = q + (((size_t)b * Hq + h) * K + k) * D;
  const float* kb = kc + ((size_t)b * Hkv + hkv) * (size_t)Lmax * D;
  const float* vb = vc + ((size_t)b * Hkv + hkv) * (size_t)D * Lmax;
  float mx = -INFINITY;
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    float s = 0.f;
    for (int d = 0; d < D; ++d) s = fmaf(qp[d], kb[(size_t)j * D + d], s);
    s *= scale;
    sc[j] = s;
    mx = fmaxf(mx, s);
  }
  red[threadIdx.x] = mx;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + w]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float sum = 0.f;
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    float p = expf(sc[j] - mx);
    sc[j] = p;
    sum += p;
  }
  red[threadIdx.x] = sum;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const float inv = 1.f / red[0];
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    const float* vr = vb + (size_t)d * Lmax;
    float acc = 0.f;
    for (int j = 0; j < n; ++j) acc = fmaf(sc[j], vr[j], acc);
    o[((size_t)b * K + k) * (Hq * D) + h * D + d] = acc * inv;
  }
}

void attention_f32(const Dims& dm, int B, int K, const int* f, const float* q, const float* kc, const float* vc,
                   int Lmax, float* o, hipStream_t st) {
  hipLaunchKernelGGL(attn_f32_kernel, dim3(K, dm.Hq, B), dim3(256), 0, st, K, dm.Hq, dm.Hkv, dm.D, Lmax, f, q, kc, vc,
                     o, 1.0f / sqrtf((float)dm.D));
}

}  // namespace ssd
