// Embedding gather, per-position correction rules and commit bookkeeping.
//
// Correction (paper Sec. 3.3, "Verification as Auto Correction"): every
// drafted position k is decided independently and in parallel, one
// workgroup per position:
//   (A) greedy  : argmax of the scoring logits (ties -> lowest code)
//   (B) sample  : inverse-CDF sample of p = softmax(top_k(logits / T))
//   (C) accept/reject: keep the token t with probability min(p(t)/q(t), 1),
//       else sample the residual [p - q]_+; a rejected position stores this
//       round's logits as its next reference q (an accepted one keeps q).
// q is the stored reference warped like p, or a point mass at t.
// Probabilities, sums and the inverse CDF are float64; the top-k set is
// found by an 8-bit radix select over order-preserving float keys, ties at
// the boundary resolved towards lower codes.  Uniforms: 24-bit SplitMix64
// outputs at a counter built from (sequence, position, round, stream)
// (Steele, Lea & Flood, OOPSLA 2014).
#include "ssd_internal.h"

namespace ssd {

__device__ __forceinline__ uint16_t f2bf_m(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ---------------- embedding ----------------
template <bool BF>
__global__ __launch_bounds__(256) void embed_kernel(const void* emb, const int* tok, int d, int V, const float* g,
                                                    float* x, void* xn, size_t xn_plane, float* ssq) {
  __shared__ float red[256];
  const int t = blockIdx.x;
  int id = tok[t];
  id = id < 0 ? 0 : (id >= V ? V - 1 : id);
  float s = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = BF ? __uint_as_float(((uint32_t)((const uint16_t*)emb)[(size_t)id * d + i]) << 16)
                 : ((const float*)emb)[(size_t)id * d + i];
    x[(size_t)t * d + i] = v;
    float gv = g[i] * v;
    if (BF) {
      // fp32 activation as hi + lo bf16 planes
      const uint16_t hi = f2bf_m(gv);
      ((uint16_t*)xn)[(size_t)t * d + i] = hi;
      ((uint16_t*)xn)[xn_plane + (size_t)t * d + i] = f2bf_m(gv - __uint_as_float((uint32_t)hi << 16));
    } else {
      ((float*)xn)[(size_t)t * d + i] = gv;
    }
    s += v * v;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) ssq[t] = red[0];
}

void embed(const Dims& dm, const void* emb, const int* tok, int M, const float* g, float* x, void* xn,
           size_t xn_plane, float* ssq, hipStream_t st) {
  if (dm.bf16)
    hipLaunchKernelGGL(embed_kernel<true>, dim3(M), dim3(256), 0, st, emb, tok, dm.d, dm.V, g, x, xn, xn_plane, ssq);
  else
    hipLaunchKernelGGL(embed_kernel<false>, dim3(M), dim3(256), 0, st, emb, tok, dm.d, dm.V, g, x, xn, xn_plane, ssq);
}

__global__ __launch_bounds__(256) void ssq_kernel(const float* x, int d, float* ssq) {
  __shared__ float red[256];
  const int t = blockIdx.x;
  float s = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float v = x[(size_t)t * d + i];
    s += v * v;
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) ssq[t] = red[0];
}

void norm_rows_f32(const float* x, int M, int d, const float* g, float* xn, float* ssq, hipStream_t st) {
  (void)g;
  (void)xn;
  hipLaunchKernelGGL(ssq_kernel, dim3(M), dim3(256), 0, st, x, d, ssq);
}

// ---------------- block helpers (256 threads) ----------------
constexpr int NT_SEL = 256;

__device__ __forceinline__ uint32_t fkey(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// output number c+1 of the SplitMix64 stream seeded with `seed`, top 24 bits in [0,1)
__device__ __forceinline__ double uniform24(unsigned long long seed, int b, int pos, unsigned round, int stream) {
  const uint64_t c = ((uint64_t)b << 44) | ((uint64_t)pos << 20) | ((uint64_t)(round & 0xFFFFu) << 4) | (uint64_t)stream;
  const uint64_t z = sm_mix(seed + (c + 1ull) * 0x9E3779B97F4A7C15ull);
  return (double)(z >> 40) * (1.0 / 16777216.0);
}

struct SelShared {
  double dred[NT_SEL / 64];
  float fred[NT_SEL / 64];
  int ired[NT_SEL / 64];
  int hist[256];
  int tie_base[NT_SEL];
  double pre[NT_SEL];
  int bc_i[4];
  double bc_d[4];
  unsigned bc_u[2];
};

__device__ double block_sum_d(double v, SelShared& sh) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh.dred[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = ((sh.dred[0] + sh.dred[1]) + sh.dred[2]) + sh.dred[3];
  __syncthreads();
  return r;
}

__device__ float block_max_f(float v, SelShared& sh) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh.fred[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = fmaxf(fmaxf(sh.fred[0], sh.fred[1]), fmaxf(sh.fred[2], sh.fred[3]));
  __syncthreads();
  return r;
}

__device__ int block_min_i(int v, SelShared& sh) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh.ired[threadIdx.x >> 6] = v;
  __syncthreads();
  int r = min(min(sh.ired[0], sh.ired[1]), min(sh.ired[2], sh.ired[3]));
  __syncthreads();
  return r;
}

__device__ int block_max_i(int v, SelShared& sh) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh.ired[threadIdx.x >> 6] = v;
  __syncthreads();
  int r = max(max(sh.ired[0], sh.ired[1]), max(sh.ired[2], sh.ired[3]));
  __syncthreads();
  return r;
}

// argmax with ties to the lowest index over row[0..V)
// Lowest index among the maxima.  Thread t scans elements 4t + 1024 j .. +3
// in ascending order (16-byte loads: each wave load is one contiguous 1 KiB
// span); the reductions below keep the lower index among equal values, so
// the result does not depend on how the elements are dealt to threads.
__device__ int block_argmax(const float* row, int V, SelShared& sh) {
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  if ((V & 3) == 0 && (((uintptr_t)row) & 15) == 0) {
    auto take = [&](const float4 x, int v) {
      if (x.x > bv || bi == 0x7fffffff) {
        bv = x.x;
        bi = v;
      }
      if (x.y > bv) {
        bv = x.y;
        bi = v + 1;
      }
      if (x.z > bv) {
        bv = x.z;
        bi = v + 2;
      }
      if (x.w > bv) {
        bv = x.w;
        bi = v + 3;
      }
    };
    // eight loads in flight, then taken in order (a load used right away is
    // waited for alone)
    constexpr int UB = 8, STR = NT_SEL * 4;
    int v = threadIdx.x * 4;
    for (; v + (UB - 1) * STR < V; v += UB * STR) {
      float4 x[UB];
#pragma unroll
      for (int u = 0; u < UB; ++u) x[u] = *(const float4*)(row + v + u * STR);
#pragma unroll
      for (int u = 0; u < UB; ++u) take(x[u], v + u * STR);
    }
    for (; v < V; v += STR) take(*(const float4*)(row + v), v);
  } else {
    for (int v = threadIdx.x; v < V; v += NT_SEL) {
      const float x = row[v];
      if (x > bv || bi == 0x7fffffff) {
        bv = x;
        bi = v;
      }
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    float ov = __shfl_xor(bv, o);
    int oi = __shfl_xor(bi, o);
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    sh.fred[threadIdx.x >> 6] = bv;
    sh.ired[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  float rv = sh.fred[0];
  int ri = sh.ired[0];
  for (int w = 1; w < NT_SEL / 64; ++w) {
    if (sh.fred[w] > rv || (sh.fred[w] == rv && sh.ired[w] < ri)) {
      rv = sh.fred[w];
      ri = sh.ired[w];
    }
  }
  __syncthreads();
  return ri;
}

// The kept set of top_k(row): keys above `thr`, plus the first `need` keys equal to
// `thr` in index order.  `all` when no truncation applies.
struct TopK {
  uint32_t thr;
  int need;
  bool all;
};

struct KeepIter {
  uint32_t thr;
  int need, rank;
  bool all;
  __device__ __forceinline__ bool next(uint32_t key) {
    if (all || key > thr) return true;
    if (key == thr) {
      bool k = rank < need;
      ++rank;
      return k;
    }
    return false;
  }
};

__device__ TopK topk_select(const float* row, int V, int top_k, SelShared& sh, int* tie_base_out) {
  TopK tk;
  tk.all = (top_k <= 0 || top_k >= V);
  tk.thr = 0;
  tk.need = 0;
  const int VPT = (V + NT_SEL - 1) / NT_SEL;
  const int lo = threadIdx.x * VPT, hi = min(lo + VPT, V);
  if (tk.all) {
    *tie_base_out = 0;
    return tk;
  }
  uint32_t prefix = 0, mask = 0;
  int remaining = top_k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    sh.hist[threadIdx.x] = 0;
    __syncthreads();
    for (int v = lo; v < hi; ++v) {
      uint32_t key = fkey(row[v]);
      if ((key & mask) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255u], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int cum = 0, dgt = 255;
      for (; dgt > 0; --dgt) {
        if (cum + sh.hist[dgt] >= remaining) break;
        cum += sh.hist[dgt];
      }
      sh.bc_i[0] = dgt;
      sh.bc_i[1] = remaining - cum;
    }
    __syncthreads();
    prefix |= (uint32_t)sh.bc_i[0] << shift;
    mask |= 0xFFu << shift;
    remaining = sh.bc_i[1];
    __syncthreads();
  }
  tk.thr = prefix;
  tk.need = remaining;
  // exclusive prefix of ties per thread, in index order
  int nt = 0;
  for (int v = lo; v < hi; ++v) nt += (fkey(row[v]) == prefix);
  sh.tie_base[threadIdx.x] = nt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int i = 0; i < NT_SEL; ++i) {
      int c = sh.tie_base[i];
      sh.tie_base[i] = acc;
      acc += c;
    }
  }
  __syncthreads();
  *tie_base_out = sh.tie_base[threadIdx.x];
  __syncthreads();
  return tk;
}

// A warped distribution p_v = [v kept] exp(z_v - mz) / Z, z = row / T.
struct Warp {
  const float* row;
  TopK tk;
  int tie_base;
  double T, mz, Z;
  __device__ __forceinline__ KeepIter iter() const { return KeepIter{tk.thr, tk.need, tie_base, tk.all}; }
};

__device__ Warp make_warp(const float* row, int V, int top_k, double T, SelShared& sh) {
  Warp w;
  w.row = row;
  int tb;
  w.tk = topk_select(row, V, top_k, sh, &tb);
  w.tie_base = tb;
  w.T = T;
  const int VPT = (V + NT_SEL - 1) / NT_SEL;
  const int lo = threadIdx.x * VPT, hi = min(lo + VPT, V);
  float mx = -INFINITY;
  for (int v = lo; v < hi; ++v) mx = fmaxf(mx, row[v]);
  mx = block_max_f(mx, sh);
  w.mz = (double)mx / T;
  double s = 0.0;
  KeepIter it = w.iter();
  for (int v = lo; v < hi; ++v) {
    float x = row[v];
    if (it.next(fkey(x))) s += exp((double)x / T - w.mz);
  }
  w.Z = block_sum_d(s, sh);
  return w;
}

// probability of one code under a warp (every thread returns the same value)
__device__ double warp_prob(const Warp& w, int t, int V, SelShared& sh) {
  const int VPT = (V + NT_SEL - 1) / NT_SEL;
  const int lo = threadIdx.x * VPT, hi = min(lo + VPT, V);
  if (t >= lo && t < hi) {
    KeepIter it = w.iter();
    double pv = 0.0;
    for (int v = lo; v <= t; ++v) {
      float x = w.row[v];
      bool k = it.next(fkey(x));
      if (v == t) pv = k ? exp((double)x / w.T - w.mz) / w.Z : 0.0;
    }
    sh.bc_d[0] = pv;
  }
  __syncthreads();
  double r = sh.bc_d[0];
  __syncthreads();
  return r;
}

// inverse CDF over per-code weights produced by `wf(v, x_p, keep_p, x_q, keep_q)`;
// smallest v with cumsum > u * total; fallback: last code of positive weight.
template <typename WF>
__device__ int block_invcdf(int V, double u, WF wf, SelShared& sh) {
  const int VPT = (V + NT_SEL - 1) / NT_SEL;
  const int lo = threadIdx.x * VPT, hi = min(lo + VPT, V);
  double s = 0.0;
  int lastpos = -1;
  wf.begin();
  for (int v = lo; v < hi; ++v) {
    double w = wf(v);
    s += w;
    if (w > 0.0) lastpos = v;
  }
  sh.pre[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double acc = 0.0;
    for (int i = 0; i < NT_SEL; ++i) {
      double c = sh.pre[i];
      sh.pre[i] = acc;
      acc += c;
    }
    sh.bc_d[1] = acc;
  }
  __syncthreads();
  const double total = sh.bc_d[1];
  const double target = u * total;
  double c = sh.pre[threadIdx.x];
  int cand = 0x7fffffff;
  wf.begin();
  for (int v = lo; v < hi; ++v) {
    c += wf(v);
    if (c > target) {
      cand = v;
      break;
    }
  }
  __syncthreads();
  int best = block_min_i(cand, sh);
  if (best == 0x7fffffff) best = block_max_i(lastpos, sh);
  return best;
}

// weights of p (normalised)
struct PW {
  const Warp* p;
  KeepIter ip;
  __device__ void begin() { ip = p->iter(); }
  __device__ double operator()(int v) {
    float x = p->row[v];
    return ip.next(fkey(x)) ? exp((double)x / p->T - p->mz) / p->Z : 0.0;
  }
};

// residual [p - q]_+ with q a warp or a point mass at `pt`
struct RW {
  const Warp* p;
  const Warp* q;  // nullptr -> point mass
  int pt;
  KeepIter ip, iq;
  __device__ void begin() {
    ip = p->iter();
    if (q) iq = q->iter();
  }
  __device__ double operator()(int v) {
    float x = p->row[v];
    double pv = ip.next(fkey(x)) ? exp((double)x / p->T - p->mz) / p->Z : 0.0;
    double qv;
    if (q) {
      float y = q->row[v];
      qv = iq.next(fkey(y)) ? exp((double)y / q->T - q->mz) / q->Z : 0.0;
    } else {
      qv = (v == pt) ? 1.0 : 0.0;
    }
    double r = pv - qv;
    return r > 0.0 ? r : 0.0;
  }
};

__global__ __launch_bounds__(NT_SEL) void select_kernel(SelectArgs a) {
  __shared__ SelShared sh;
  const int k = blockIdx.x, b = blockIdx.y;
  const int V = a.Vimg;
  const size_t idx = (size_t)b * a.K + k;
  if (k < a.n_fixed ||
      (a.eol_period > 0 && (a.f[b] + k - a.eol_base) % a.eol_period == a.eol_period - 1)) {
    if (threadIdx.x == 0) a.accept[idx] = 0;  // fixed: already chosen, or an end-of-line token
    return;
  }
  const float* L = (k == 0) ? a.carry + (size_t)b * V : a.logits + (idx - 1) * V;
  int t = a.tokens[idx] - a.img_lo;
  t = t < 0 ? 0 : (t >= V ? V - 1 : t);
  const int pos = a.f[b] + k;
  int newt = t;
  bool acc = false;
  if (a.rule == SSD_GREEDY || a.truncate) {
    newt = block_argmax(L, V, sh);
    acc = (newt == t);
    if (a.truncate && threadIdx.x == 0) a.amax[idx] = newt;
  } else {
    Warp p = make_warp(L, V, a.top_k, a.temperature, sh);
    if (a.rule == SSD_SAMPLE) {
      const double u1 = uniform24(a.seed, b, pos, a.round, 1);
      PW wf{&p, KeepIter{}};
      newt = block_invcdf(V, u1, wf, sh);
      acc = (newt == t);
    } else {
      const int slot = pos % a.ring;
      const bool has_ref = a.ref_flag[(size_t)b * a.ring + slot] != 0;
      float* refrow = a.ref + ((size_t)b * a.ring + slot) * V;
      Warp q;
      double qt = 1.0;
      if (has_ref) {
        q = make_warp(refrow, V, a.top_k, a.temperature, sh);
        qt = warp_prob(q, t, V, sh);
      }
      const double pt = warp_prob(p, t, V, sh);
      const double alpha = qt > 0.0 ? fmin(pt / qt, 1.0) : (pt > 0.0 ? 1.0 : 0.0);
      const double u0 = uniform24(a.seed, b, pos, a.round, 0);
      if (u0 < alpha) {
        acc = true;
      } else {
        RW wf{&p, has_ref ? &q : nullptr, t, KeepIter{}, KeepIter{}};
        // total residual mass (same association as the inverse CDF's)
        const double u1 = uniform24(a.seed, b, pos, a.round, 1);
        // zero residual (rounding only): keep the token
        double s = 0.0;
        {
          const int VPT = (V + NT_SEL - 1) / NT_SEL;
          const int lo = threadIdx.x * VPT, hi = min(lo + VPT, V);
          wf.begin();
          for (int v = lo; v < hi; ++v) s += wf(v);
        }
        const double tot = block_sum_d(s, sh);
        if (!(tot > 0.0)) {
          acc = true;
        } else {
          newt = block_invcdf(V, u1, wf, sh);
          acc = false;
          // the rejected position's reference becomes this round's backbone logits
          for (int v = threadIdx.x; v < V; v += NT_SEL) refrow[v] = L[v];
          if (threadIdx.x == 0) a.ref_flag[(size_t)b * a.ring + slot] = 1;
        }
      }
    }
  }
  if (threadIdx.x == 0) {
    a.tokens[idx] = newt + a.img_lo;
    a.accept[idx] = acc ? 1 : 0;
    if (acc) atomicAdd(&a.count[b], 1);
  }
}

void select_tokens(const SelectArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(a.K, a.B), dim3(NT_SEL), 0, st, a);
}

// truncate mode: accepted run, new frontier and carry
__global__ __launch_bounds__(256) void truncate_kernel(SelectArgs a, int* f, float* carry) {
  __shared__ int kk_s;
  const int b = blockIdx.x;
  if (threadIdx.x == 0) {
    int kk = a.n_fixed;
    while (kk < a.K && a.accept[(size_t)b * a.K + kk]) ++kk;
    kk_s = kk;
    a.count[b] = kk - a.n_fixed;
  }
  __syncthreads();
  const int kk = kk_s;
  if (kk >= 1) {
    const float* src = a.logits + ((size_t)b * a.K + kk - 1) * a.Vimg;
    for (int v = threadIdx.x; v < a.Vimg; v += 256) carry[(size_t)b * a.Vimg + v] = src[v];
  }
  __syncthreads();
  if (threadIdx.x == 0) f[b] += kk;
}

void truncate_finalize(const SelectArgs& a, int* f, hipStream_t st) {
  hipLaunchKernelGGL(truncate_kernel, dim3(a.B), dim3(256), 0, st, a, f, (float*)a.carry);
}

// commit: carry <- logits row (b * rps + last); f += f_inc; drop the references of the committed positions
// Workgroups (x, b): the carry row of sequence b is copied by all gridDim.x
// workgroups of b in 16-byte vectors; workgroup 0 alone clears the reference
// flags of the committed positions and advances the frontier.
__global__ __launch_bounds__(256) void commit_kernel(int Vimg, const float* logits, int rps, int last, float* carry,
                                                     int* f, int f_inc, int* ref_flag, int ring) {
  const int b = blockIdx.y;
  const float* src = logits + ((size_t)b * rps + last) * Vimg;
  float* dst = carry + (size_t)b * Vimg;
  if ((Vimg & 3) == 0) {
    for (int v = (blockIdx.x * 256 + threadIdx.x) * 4; v < Vimg; v += gridDim.x * 1024)
      *(float4*)(dst + v) = *(const float4*)(src + v);
  } else {
    for (int v = blockIdx.x * 256 + threadIdx.x; v < Vimg; v += gridDim.x * 256) dst[v] = src[v];
  }
  if (blockIdx.x != 0) return;
  const int f0 = f[b];
  if (ref_flag)
    for (int k = threadIdx.x; k < f_inc && k < ring; k += 256) ref_flag[(size_t)b * ring + (f0 + k) % ring] = 0;
  __syncthreads();
  if (threadIdx.x == 0) f[b] = f0 + f_inc;
}

// workgroups per sequence: one per 1024 carry values, at most 16
static int commit_groups(int Vimg) { return std::max(1, std::min(16, (Vimg + 1023) / 1024)); }

void commit_update(int B, int K, int Vimg, const float* logits, float* carry, int* f, int* ref_flag, int ring,
                   hipStream_t st) {
  // K > 0: logits rows are [B][K], carry from row K-1, f += K.
  // K < 0: logits rows are [B][1] (last row only), f += -K.
  int rps = K > 0 ? K : 1, last = K > 0 ? K - 1 : 0, inc = K > 0 ? K : -K;
  hipLaunchKernelGGL(commit_kernel, dim3(commit_groups(Vimg), B), dim3(256), 0, st, Vimg, logits, rps, last, carry, f,
                     inc, ref_flag, ring);
}

void commit_prefix(int B, int rps, int Kc, int Vimg, const float* logits, float* carry, int* f, int* ref_flag,
                   int ring, hipStream_t st) {
  hipLaunchKernelGGL(commit_kernel, dim3(commit_groups(Vimg), B), dim3(256), 0, st, Vimg, logits, rps, Kc - 1, carry,
                     f, Kc, ref_flag, ring);
}

// Classifier-free guidance: guided logits l_u + w (l_c - l_u) of each image b
// (conditional stream b, unconditional stream Bi + b).  Workgroup (r, b): rows
// r < K of the pass's logits [2*Bi*K][V] (row = stream * K + r), r = K the
// carry [2*Bi][V].  K = 0 mixes the carry only.
__global__ __launch_bounds__(256) void cfg_mix_kernel(int Bi, int K, int Vimg, float w, const float* logits,
                                                      const float* carry, float* out_logits, float* out_carry) {
  const int r = blockIdx.x, b = blockIdx.y;
  const float *c, *u;
  float* o;
  if (r < K) {
    c = logits + ((size_t)b * K + r) * Vimg;
    u = logits + ((size_t)(Bi + b) * K + r) * Vimg;
    o = out_logits + ((size_t)b * K + r) * Vimg;
  } else {
    c = carry + (size_t)b * Vimg;
    u = carry + (size_t)(Bi + b) * Vimg;
    o = out_carry + (size_t)b * Vimg;
  }
  if ((Vimg & 3) == 0) {
    const float4* c4 = reinterpret_cast<const float4*>(c);
    const float4* u4 = reinterpret_cast<const float4*>(u);
    float4* o4 = reinterpret_cast<float4*>(o);
    for (int v = threadIdx.x; v < Vimg / 4; v += 256) {
      const float4 x = c4[v], y = u4[v];
      o4[v] = make_float4(y.x + w * (x.x - y.x), y.y + w * (x.y - y.y), y.z + w * (x.z - y.z), y.w + w * (x.w - y.w));
    }
  } else {
    for (int v = threadIdx.x; v < Vimg; v += 256) o[v] = u[v] + w * (c[v] - u[v]);
  }
}

void cfg_mix(int Bi, int K, int Vimg, float w, const float* logits, const float* carry, float* out_logits,
             float* out_carry, hipStream_t st) {
  hipLaunchKernelGGL(cfg_mix_kernel, dim3(K + 1, Bi), dim3(256), 0, st, Bi, K, Vimg, w, logits, carry, out_logits,
                     out_carry);
}

// Which XCD (accelerator complex die) each workgroup runs on: the XCC_ID
// hardware register (bits [3:0]).  Used once at start-up to verify the
// round-robin workgroup-to-XCD dispatch the split-K reductions rely on.
__global__ void xcc_probe_kernel(int* out) {
  if (threadIdx.x == 0) out[blockIdx.x] = (int)(__builtin_amdgcn_s_getreg(20 | (0 << 6) | ((4 - 1) << 11)) & 0xF);
}

void xcc_probe(int* out, int n_wg, hipStream_t st) {
  hipLaunchKernelGGL(xcc_probe_kernel, dim3(n_wg), dim3(64), 0, st, out);
}

__global__ void fill_u32_kernel(unsigned* p, size_t n, unsigned v) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

void fill_u32(unsigned* p, size_t n, unsigned v, hipStream_t st) {
  if (n == 0) return;
  hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n, v);
}

// rows of src [B][K][Vimg] become the references of positions f+k (only_new: keep existing ones)
__global__ __launch_bounds__(256) void set_ref_kernel(int rows_per_b, int Vimg, const float* src, const int* f,
                                                      float* ref, int* ref_flag, int ring, int only_new) {
  const int k = blockIdx.x, b = blockIdx.y;
  const int slot = (f[b] + k) % ring;
  int* fl = ref_flag + (size_t)b * ring + slot;
  if (only_new && *fl) return;
  const float* s = src + ((size_t)b * rows_per_b + k) * Vimg;
  float* d = ref + ((size_t)b * ring + slot) * Vimg;
  for (int v = threadIdx.x; v < Vimg; v += 256) d[v] = s[v];
  __syncthreads();
  if (threadIdx.x == 0) *fl = 1;
}

void set_ref_rows(int B, int K, int rows_per_b, int Vimg, const float* src, const int* f, float* ref, int* ref_flag,
                  int ring, int only_new, hipStream_t st) {
  hipLaunchKernelGGL(set_ref_kernel, dim3(K, B), dim3(256), 0, st, rows_per_b, Vimg, src, f, ref, ref_flag, ring,
                     only_new);
}

// first image token from the carry: argmax (rule A) or a sample of the warped carry (uniform stream 2, round 0)
__global__ __launch_bounds__(NT_SEL) void first_token_kernel(int Vimg, int img_lo, const float* carry, int rule, int top_k,
                                                              double T, unsigned long long seed, const int* f,
                                                              int* out_abs, int out_stride) {
  __shared__ SelShared sh;
  const int b = blockIdx.x;
  const float* L = carry + (size_t)b * Vimg;
  int v;
  if (rule == SSD_GREEDY) {
    v = block_argmax(L, Vimg, sh);
  } else {
    Warp p = make_warp(L, Vimg, top_k, T, sh);
    const double u1 = uniform24(seed, b, f[b], 0u, 2);
    PW wf{&p, KeepIter{}};
    v = block_invcdf(Vimg, u1, wf, sh);
  }
  if (threadIdx.x == 0) out_abs[(size_t)b * out_stride] = v + img_lo;
}

// Draft-head input z = [h; e] as split bf16 planes [R][2d]: h fp32 (hi/lo),
// e the bf16 embedding row of the token (exact in the hi plane).
__global__ __launch_bounds__(256) void draft_input_kernel(const float* h, const uint16_t* emb, const int* tok, int d,
                                                          uint16_t* z, size_t plane) {
  const int r = blockIdx.x;
  const float* hr = h + (size_t)r * d;
  const uint16_t* er = emb + (size_t)tok[r] * d;
  uint16_t* zr = z + (size_t)r * 2 * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    const float v = hr[i];
    const uint16_t hi = f2bf_m(v);
    zr[i] = hi;
    zr[plane + i] = f2bf_m(v - __uint_as_float((uint32_t)hi << 16));
    zr[d + i] = er[i];
    zr[plane + d + i] = 0;
  }
}

void draft_input(const float* h, const void* emb, const int* tok, int R, int d, void* z, size_t plane,
                 hipStream_t st) {
  hipLaunchKernelGGL(draft_input_kernel, dim3(R), dim3(256), 0, st, h, (const uint16_t*)emb, tok, d, (uint16_t*)z,
                     plane);
}

// fp32 models: z = [h; e] as plain fp32 rows [R][2d]
__global__ __launch_bounds__(256) void draft_input_f32_kernel(const float* h, const float* emb, const int* tok, int d,
                                                              float* z) {
  const int r = blockIdx.x;
  const float* hr = h + (size_t)r * d;
  const float* er = emb + (size_t)tok[r] * d;
  float* zr = z + (size_t)r * 2 * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    zr[i] = hr[i];
    zr[d + i] = er[i];
  }
}

void draft_input_f32(const float* h, const float* emb, const int* tok, int R, int d, float* z, hipStream_t st) {
  hipLaunchKernelGGL(draft_input_f32_kernel, dim3(R), dim3(256), 0, st, h, emb, tok, d, z);
}

void first_token(int B, int Vimg, int img_lo, const float* carry, int rule, int top_k, double temperature,
                 unsigned long long seed, const int* f, int* out_abs, int out_stride, hipStream_t st) {
  hipLaunchKernelGGL(first_token_kernel, dim3(B), dim3(NT_SEL), 0, st, Vimg, img_lo, carry, rule, top_k, temperature,
                     seed, f, out_abs, out_stride);
}

// The greedy argmax a of a logits row (lowest code among equal maxima) placed
// at image index x = f[b] - P + pos_off of sequence b: with `keep` it is a
// planted draft (a where keep[x] is set, else the other code
// repl[x] + (repl[x] >= a)), without it the token itself (the pending token of
// strict verification).  `active` (optional) gates sequences: an inactive one
// is skipped, and a planted replacement (or x outside [0, x_end)) deactivates
// it.  One workgroup per sequence.
__global__ __launch_bounds__(NT_SEL) void place_argmax_kernel(PlaceArgs a) {
  __shared__ SelShared sh;
  const int b = blockIdx.x;
  if (a.active && a.active[b] == 0) return;
  const int x = a.f[b] - a.P + a.pos_off;
  if (x < 0 || x >= a.x_end) {
    if (a.active && threadIdx.x == 0) a.active[b] = 0;
    return;
  }
  const int am = block_argmax(a.logits + (size_t)b * a.row_stride, a.Vimg, sh);
  int t = am;
  bool kept = true;
  if (a.keep) {
    kept = a.keep[(size_t)b * a.x_end + x] != 0;
    if (!kept) {
      const int r = a.repl[(size_t)b * a.x_end + x];
      t = r + (r >= am ? 1 : 0);
    }
  }
  if (threadIdx.x == 0) {
    const int id = t + a.img_lo;
    a.img[(size_t)b * a.img_stride + x] = id;
    if (a.table) a.table[(size_t)b * a.x_end + x] = id;
    if (a.next_tok) a.next_tok[b] = id;
    if (a.active && !kept) a.active[b] = 0;
  }
}

void place_argmax(const PlaceArgs& a, int B, hipStream_t st) {
  hipLaunchKernelGGL(place_argmax_kernel, dim3(B), dim3(NT_SEL), 0, st, a);
}

// tok[b][k] = img[b][f[b] - P + k], k < K (blocks at per-sequence frontiers)
__global__ __launch_bounds__(64) void gather_block_kernel(const int* img, int img_stride, const int* f, int P, int K,
                                                          int* tok) {
  const int b = blockIdx.x;
  const int* src = img + (size_t)b * img_stride + (f[b] - P);
  for (int k = threadIdx.x; k < K; k += 64) tok[(size_t)b * K + k] = src[k];
}

void gather_block(const int* img, int img_stride, const int* f, int P, int K, int B, int* tok, hipStream_t st) {
  hipLaunchKernelGGL(gather_block_kernel, dim3(B), dim3(64), 0, st, img, img_stride, f, P, K, tok);
}

__global__ void add_i32_kernel(int* p, int n, int delta) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] += delta;
}

void add_i32(int* p, int n, int delta, hipStream_t st) {
  if (n <= 0 || delta == 0) return;
  hipLaunchKernelGGL(add_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, st, p, n, delta);
}

}  // namespace ssd
