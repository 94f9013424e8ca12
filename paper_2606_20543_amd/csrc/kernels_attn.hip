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
#include "tiles.h"

namespace ssd {

// key split: one wave per SIMD, so the register file holds two K/V blocks,
// the queries and the accumulators without the compiler sinking the prefetch
// loads
template <int D, int QPW>
__global__ __launch_bounds__(AtShape<QPW>::THREADS) __attribute__((amdgpu_waves_per_eu(1, 1)))
void attn_bf16_kernel(AttnKArgs a) {
  constexpr int NW = AtShape<QPW>::WAVES, ROWS = QPW * 16, RS = D + 4;
  __shared__ __align__(16) float sm_o[NW * ROWS * RS];
  __shared__ float sm_m[NW * ROWS], sm_l[NW * ROWS];
  __shared__ int is_last;
  attn_unit<D, QPW, PlainMem, true, PlainMem, false, false>(a, blockIdx.x, sm_o, sm_m, sm_l, &is_last);
}

// query split: two workgroups per CU, so each SIMD runs waves of two
// workgroups that meet no common barrier (at most 256 registers each; the
// K/V stages and the output stage share their LDS bytes, used one after the
// other, 68 KB per workgroup)
template <int D, int QPW>
__global__ __launch_bounds__(AtShape<QPW>::THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_qs_kernel(AttnKArgs a) {
  constexpr int NW = AtShape<QPW>::WAVES, ROWS = QPW * 16, RS = D + 4;
  constexpr int O_BYTES = NW * ROWS * RS * 4, KV_BYTES = AT_KV_STAGES * at_kv_tiles<D>() * 1024;
  __shared__ __align__(16) char sm_u[O_BYTES > KV_BYTES ? O_BYTES : KV_BYTES];
  __shared__ float sm_m[NW * ROWS], sm_l[NW * ROWS];
  __shared__ int is_last;
  attn_unit<D, QPW, PlainMem, true, PlainMem, false, true>(a, blockIdx.x, (float*)sm_u, sm_m, sm_l, &is_last,
                                                           nullptr, (uint16_t*)sm_u);
}

AttnPlan attn_plan(const Dims& dm, int B, int K, int max_ctx_now, int xcd, int grid) {
  AttnPlan p;
  p.xcd = xcd;
  const int g = dm.Hq / dm.Hkv;
  p.rows = K * g;
  const int qt = (p.rows + 15) / 16;
  p.qpw = (qt >= 4 && grid == 0) ? 2 : 1;
  // 128 or more query rows per (sequence, KV head): the waves split the rows,
  // so a K/V block is streamed once per 128 rows instead of once per 32
  p.qs = (qt >= 8 && grid == 0 && dm.D == 128) ? 1 : 0;  // (with D = 64 its chunk statistics outgrow the LDS stage)
  p.nqg = (qt + (p.qs ? 4 : 1) * p.qpw - 1) / ((p.qs ? 4 : 1) * p.qpw);
  const long units = (long)B * dm.Hkv * p.nqg;
  const int ctx = max_ctx_now < 1 ? 1 : max_ctx_now;
  auto chunk_for = [&](int n) {  // whole workgroup steps covering ctx in n chunks
    const int per = (ctx + n - 1) / n;
    return ((per + AT_STEP - 1) / AT_STEP) * AT_STEP;
  };
  int best = 1;
  const long slots = grid > 0 ? grid : (p.qs ? 512 : 256);  // query split: two workgroups per CU
  if (units >= slots) {
    // many query groups: the chip is full, chunks only bound the per-workgroup stream
    int chunk = AT_STEP;
    while ((chunk < 16 * AT_STEP && units * ((ctx + chunk - 1) / chunk) > 1024) ||
           (ctx + chunk - 1) / chunk > AT_MAX_CHUNKS)
      chunk *= 2;
    p.chunk = chunk;
  } else {
    // few query groups: a chunk costs about 0.85 us per 128-key step of its
    // workgroup (per 32-key step when the waves split the query rows), a split
    // adds the partial publish and the merge (about 1.6 us + 0.08 us per
    // chunk); measured on MI355X with D = 128
    const double keys_per_step = p.qs ? AT_KEYS : AT_STEP;
    double best_t = 1e30;
    for (int n = 1;
         n <= AT_MAX_CHUNKS && (grid > 0 ? (long)xcd_grid(B * dm.Hkv, p.nqg * n, xcd) : units * n) <= slots; ++n) {
      const int ch = chunk_for(n);
      const int nn = (ctx + ch - 1) / ch;
      if (nn != n) continue;
      const double t = 0.85 * (ch / keys_per_step) * (dm.D / 128.0) + (n > 1 ? 1.6 + 0.08 * n : 0.0);
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
  return (size_t)B * dm.Hkv * p.nqg * p.nchunk * p.group_rows() * (dm.D + 2);
}

template <int D, int QPW, bool QS = false>
static void launch_attn(const AttnKArgs& a, hipStream_t st) {
  if constexpr (QS)
    launch_timed(attn_qs_kernel<D, QPW>, dim3(attn_items(a)), dim3(AtShape<QPW>::THREADS), st, a);
  else
    launch_timed(attn_bf16_kernel<D, QPW>, dim3(attn_items(a)), dim3(AtShape<QPW>::THREADS), st, a);
}

AttnKArgs attn_args(const Dims& dm, const AttnPlan& p, int B, int K, const int* f, const void* q, size_t q_plane,
                    const void* kc, const void* vc, int Lmax, void* o, size_t o_plane, float* partials,
                    unsigned* counters) {
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
  a.spart = (float2*)(partials + (size_t)a.groups * p.nchunk * p.group_rows() * dm.D);
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
  return a;
}

int attn_items(const AttnKArgs& a) {
  return xcd_grid(a.heads, a.nqg * a.nchunk, a.xcd);
}

void attention_bf16(const Dims& dm, const AttnPlan& p, int B, int K, const int* f, const void* q, size_t q_plane,
                    const void* kc, const void* vc, int Lmax, void* o, size_t o_plane, float* partials,
                    unsigned* counters, hipStream_t st) {
  const AttnKArgs a = attn_args(dm, p, B, K, f, q, q_plane, kc, vc, Lmax, o, o_plane, partials, counters);
  if (dm.D == 128) {
    if (p.qs) launch_attn<128, 2, true>(a, st);
    else if (p.qpw == 2) launch_attn<128, 2>(a, st);
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
