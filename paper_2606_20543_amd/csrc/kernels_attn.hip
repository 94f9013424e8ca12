// Block-causal multi-query attention of the verify pass over the KV cache.
//
// A block of K tokens at positions [f, f+K) attends under the backbone's
// ordinary causal mask over raster positions: block token k (position f+k)
// sees cache slots [0, f+k].  The paper's backbone is used unmodified
// (Sec. 3.3), so no other mask exists; the drafted block simply occupies the
// next raster positions.
//
// bf16 path: a workgroup of four waves owns one key chunk of one query group
// (up to 32 query rows of one sequence x KV head; the K*g rows of a KV head,
// g = query heads per KV head, are tiled by 16).  Wave w streams the chunk's
// 32-key blocks w, w+4, ... : S^T = K Q^T and O^T = V^T P^T run on
// v_mfma_f32_16x16x32_bf16 with queries as the MFMA columns, so the softmax
// statistics of a query live in one lane column and need two cross-lane
// shuffles; the P^T operand is built in registers straight from the S^T
// accumulators (its key order is matched by reading the transposed V cache),
// so P never touches LDS.  The four waves' (max, sum, O) triples are merged
// through LDS.  Chunks of one query group run on workgroups of one XCD; each
// publishes its merged triple and the last to arrive combines them in chunk
// order, all threads loading in parallel.
#include "ssd_internal.h"

namespace ssd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t f2bf_a(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

constexpr int ATTN_WAVES = 4;
constexpr int ATTN_KEYS = 32;                           // keys per wave step
constexpr int ATTN_MIN_CHUNK = ATTN_WAVES * ATTN_KEYS;  // keys per workgroup step
constexpr int ATTN_MAX_CHUNKS = 64;

struct AttnKArgs {
  const uint16_t* q;   // [B][Hq][K][D], hi plane then lo plane (q_plane elements apart)
  const uint16_t* kc;  // [B][Hkv][Lmax][D]
  const uint16_t* vc;  // [B][Hkv][D][Lmax]
  uint16_t* o;         // [B*K][Hq*D], hi plane then lo plane (o_plane elements apart)
  size_t q_plane, o_plane;
  float* opart;        // [groups][nchunk][QPW*16][D]   chunk partial O (relative to the chunk max)
  float2* spart;       // [groups][nchunk][QPW*16]      chunk (max, sum), log2 domain
  unsigned* counters;  // [groups]
  const int* f;
  int K, Hq, Hkv, g, Lmax, rows, chunk, nchunk, nqg, groups, xcd;
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

template <int D, int QPW>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnKArgs a) {
  constexpr int KD = D / 32;   // 32-wide k steps over the head dimension
  constexpr int DT = D / 16;   // 16-row d tiles of O^T
  constexpr int ROWS = QPW * 16;
  constexpr int RS = D + 4;    // LDS row stride (floats): rows of one wave fall on different banks
  constexpr int NV = ROWS * D / 4 / 256;  // float4 outputs per thread
  static_assert(NV >= 1 && ROWS * D / 4 == NV * 256, "thread map");
  static_assert(3 * ATTN_MAX_CHUNKS * ROWS <= ATTN_WAVES * ROWS * RS, "chunk statistics fit the O stage");
  __shared__ __align__(16) float sm_o[ATTN_WAVES * ROWS * RS];
  __shared__ float sm_m[ATTN_WAVES * ROWS], sm_l[ATTN_WAVES * ROWS];
  __shared__ int is_last;

  // reduction group = (sequence x KV head, query group); members = key chunks, all on one XCD
  int grp_id, c;
  xcd_unmap(blockIdx.x, a.nchunk, a.xcd, grp_id, c);
  if (grp_id >= a.groups) return;
  const int qg = grp_id % a.nqg, z = grp_id / a.nqg;
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

  // query fragments (B operand of S^T = K Q^T): lane holds row col of tile qt, d = 8*grp.. (+32 kd);
  // q is fp32 carried as hi + lo bf16 operands
  bf16x8 qh[QPW][KD], ql[QPW][KD];
  int qpos[QPW];
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    const int r = rbase + qt * 16 + col;
    const bool ok = r < a.rows;
    const int j = ok ? r / a.K : 0, k = ok ? r - (r / a.K) * a.K : 0;
    qpos[qt] = ok ? fb + k : -1;
    const uint16_t* qp = a.q + (((size_t)b * a.Hq + hkv * a.g + j) * a.K + k) * D + grp * 8;
#pragma unroll
    for (int kd = 0; kd < KD; ++kd) {
      uint4 vh = ok ? *(const uint4*)(qp + kd * 32) : make_uint4(0, 0, 0, 0);
      uint4 vl = ok ? *(const uint4*)(qp + a.q_plane + kd * 32) : make_uint4(0, 0, 0, 0);
      qh[qt][kd] = __builtin_bit_cast(bf16x8, vh);
      ql[qt][kd] = __builtin_bit_cast(bf16x8, vl);
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

  const uint16_t* kbase = a.kc + ((size_t)b * a.Hkv + hkv) * a.Lmax * D;
  const uint16_t* vbase = a.vc + ((size_t)b * a.Hkv + hkv) * (size_t)D * a.Lmax;

  for (int key0 = kbeg + wave * ATTN_KEYS; key0 < kend; key0 += ATTN_MIN_CHUNK) {
    // S^T tiles for keys key0 + [0,16) and key0 + [16,32)
    floatx4 s[2][QPW];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      int krow = key0 + kt * 16 + col;
      krow = krow < a.Lmax ? krow : a.Lmax - 1;
      const uint16_t* kp = kbase + (size_t)krow * D + grp * 8;
      bf16x8 kf[KD];
#pragma unroll
      for (int kd = 0; kd < KD; ++kd) kf[kd] = __builtin_bit_cast(bf16x8, *(const uint4*)(kp + kd * 32));
#pragma unroll
      for (int qt = 0; qt < QPW; ++qt) {
        floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kd = 0; kd < KD; ++kd) {
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kd], qh[qt][kd], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[kd], ql[qt][kd], acc, 0, 0, 0);
        }
        s[kt][qt] = acc;
      }
    }
    // V^T fragments: lane row d = dt*16 + col, keys key0 + 4*grp + [0,4) and key0 + 16 + 4*grp + [0,4)
    bf16x8 vf[DT];
    {
      int kA = key0 + 4 * grp, kB = key0 + 16 + 4 * grp;
      kA = kA + 3 < a.Lmax ? kA : a.Lmax - 4;
      kB = kB + 3 < a.Lmax ? kB : a.Lmax - 4;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const uint16_t* vp = vbase + (size_t)(dt * 16 + col) * a.Lmax;
        uint2 lo = *(const uint2*)(vp + kA);
        uint2 hi = *(const uint2*)(vp + kB);
        uint4 v = make_uint4(lo.x, lo.y, hi.x, hi.y);
        vf[dt] = __builtin_bit_cast(bf16x8, v);
      }
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
          float v = s[kt][qt][e] * a.scale_log2;
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
        float p = none ? 0.f : exp2f(sv[i] - mnew);
        ps += p;
        pb[i] = f2bf_a(p);
        pl[i] = f2bf_a(p - __uint_as_float((uint32_t)pb[i] << 16));
      }
      l[qt] = l[qt] * alpha + ps;
      m[qt] = mnew;
      uint4 pv, pw;
      pv.x = (uint32_t)pb[0] | ((uint32_t)pb[1] << 16);
      pv.y = (uint32_t)pb[2] | ((uint32_t)pb[3] << 16);
      pv.z = (uint32_t)pb[4] | ((uint32_t)pb[5] << 16);
      pv.w = (uint32_t)pb[6] | ((uint32_t)pb[7] << 16);
      pw.x = (uint32_t)pl[0] | ((uint32_t)pl[1] << 16);
      pw.y = (uint32_t)pl[2] | ((uint32_t)pl[3] << 16);
      pw.z = (uint32_t)pl[4] | ((uint32_t)pl[5] << 16);
      pw.w = (uint32_t)pl[6] | ((uint32_t)pl[7] << 16);
      bf16x8 pf = __builtin_bit_cast(bf16x8, pv);
      bf16x8 pg = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        O[qt][dt] *= alpha;
        O[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[dt], pf, O[qt][dt], 0, 0, 0);
        O[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[dt], pg, O[qt][dt], 0, 0, 0);
      }
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

  // merge the four waves: thread owns NV float4 slots (row r, dims 4*d4..)
  floatx4 acc[NV];
  float Lr[NV], Mr[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int idx = threadIdx.x + 256 * i;
    const int r = idx / (D / 4), d4 = idx - r * (D / 4);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < ATTN_WAVES; ++w) M = fmaxf(M, sm_m[w * ROWS + r]);
    float L = 0.f;
    floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < ATTN_WAVES; ++w) {
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
      const int idx = threadIdx.x + 256 * i;
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
      const int idx = threadIdx.x + 256 * i;
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
  float* cm = sm_o;                          // [nch][ROWS] chunk max
  float* cl = sm_o + ATTN_MAX_CHUNKS * ROWS; // [nch][ROWS] chunk sum, then weight
  for (int i = threadIdx.x; i < nch * ROWS; i += 256) {
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
  const floatx4* G = (const floatx4*)(a.opart + gbase * ROWS * D);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int idx = threadIdx.x + 256 * i;
    const int r = idx / (D / 4), d4 = idx - r * (D / 4);
    floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int cc = 0; cc < nch; ++cc) v += G[(size_t)cc * (ROWS * D / 4) + idx] * cl[cc * ROWS + r];
    const int rg = rbase + r;
    if (rg >= a.rows) continue;
    const int j = rg / a.K, k = rg - j * a.K;
    uint16_t* op = a.o + ((size_t)b * a.K + k) * (a.Hq * D) + (hkv * a.g + j) * D + 4 * d4;
    store_split4(op, a.o_plane, v * (1.f / sm_l[r]));
  }
  if (threadIdx.x == 0) a.counters[grp_id] = 0u;
}

AttnPlan attn_plan(const Dims& dm, int B, int K, int max_ctx_now, int xcd) {
  AttnPlan p;
  p.xcd = xcd;
  const int g = dm.Hq / dm.Hkv;
  p.rows = K * g;
  const int qt = (p.rows + 15) / 16;
  p.qpw = qt >= 2 ? 2 : 1;
  p.nqg = (qt + p.qpw - 1) / p.qpw;
  // chunk (multiple of one workgroup step): enough workgroups to cover the
  // chip, at most ATTN_MAX_CHUNKS chunks per query group
  const long units = (long)B * dm.Hkv * p.nqg;
  int chunk = ATTN_MIN_CHUNK;
  auto nchunks = [&](int ch) { return (max_ctx_now + ch - 1) / ch; };
  while ((chunk < 4096 && units * nchunks(chunk) > 1024) || nchunks(chunk) > ATTN_MAX_CHUNKS) chunk *= 2;
  p.chunk = chunk;
  p.nchunk = nchunks(chunk);
  return p;
}

size_t attn_partials_floats(const Dims& dm, const AttnPlan& p, int B) {
  return (size_t)B * dm.Hkv * p.nqg * p.nchunk * p.qpw * 16 * (dm.D + 2);
}

template <int D, int QPW>
static void launch_attn(const AttnKArgs& a, hipStream_t st) {
  launch_timed(attn_bf16_kernel<D, QPW>, dim3(xcd_grid(a.groups, a.nchunk, a.xcd)), dim3(256), st, a);
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
  a.groups = B * dm.Hkv * p.nqg;
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
  a.chunk = p.chunk;
  a.nchunk = p.nchunk;
  a.nqg = p.nqg;
  a.xcd = p.nchunk > 1 ? p.xcd : 0;
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
