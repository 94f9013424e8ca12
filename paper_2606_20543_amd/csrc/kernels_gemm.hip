// Projection GEMMs of the backbone forward pass, y[t][n] = sum_k in[t][k] W[n][k],
// with the epilogues the verify step needs fused into the final write:
//   QKV    : 1/rms scale, rotary embedding at the token's raster position,
//            q to the query buffer, k/v (bf16) into the KV cache slots [f, f+K)
//   RESID  : x += y; xn = g_next * x; per-block sums of x^2 for the next 1/rms
//   SWIGLU : h = silu(gate / rms) * (up / rms)
//   LOGITS : logits = y / rms  (fp32)
//
// bf16 path (gfx950 MFMA v_mfma_f32_16x16x32_bf16): the verify step runs at
// small M (the draft count, 8..512 tokens), so the GEMMs stream the weights
// from HBM once: each wave streams its own 16-feature tiles (prepacked so one
// 16-byte load per lane fetches a whole A operand), the token rows of the
// current K-chunk sit in LDS (B operand, shared by the four waves), and the
// A loads of the next chunk are in flight while the current one is
// multiplied.  Activations arrive as hi/lo bf16 planes (fp32 precision), so
// each A tile meets two B operands.  When N/64 feature blocks cannot fill
// 256 CUs the K range is split; the last workgroup of a feature block sums
// the partials in split order (deterministic) and runs the epilogue.
#include "tiles.h"

namespace ssd {

// stored state: bf16 for bf16 models (KV cache)
template <bool BF>
__device__ __forceinline__ void st_state(void* base, size_t i, float v) {
  if (BF)
    ((uint16_t*)base)[i] = f2bf(v);
  else
    ((float*)base)[i] = v;
}

// activation: hi/lo bf16 planes for bf16 models, fp32 otherwise
template <bool BF>
__device__ __forceinline__ void st_split(void* base, size_t plane, size_t i, float v) {
  if (BF) {
    uint16_t hi = f2bf(v);
    ((uint16_t*)base)[i] = hi;
    ((uint16_t*)base)[plane + i] = f2bf(v - bf2f(hi));
  } else {
    ((float*)base)[i] = v;
  }
}

__device__ __forceinline__ float rms_scale(const EpiArgs& e, int t) {
  if (!e.ssq) return 1.f;
  float s = 0.f;
  const size_t c = (size_t)e.ssq_off + (size_t)t * e.ssq_step;
  for (int p = 0; p < e.ssq_parts; ++p) s += e.ssq[(size_t)p * e.ssq_ld + c];
  return 1.0f / sqrtf(s * e.inv_d + e.eps);
}

// Epilogue of the output pair (n, n+1), n even, for token t with accumulators
// (v0, v1) and rms scale r.  Returns the squared new residual values (RESID).
template <bool BF>
__device__ __forceinline__ float epi_pair(const EpiArgs& e, int t, int n, float v0, float v1, float r) {
  switch (e.kind) {
    case EPI_QKV: {
      const int b = t / e.Kblk, k = t - b * e.Kblk;
      const int pos = e.f[b] + k;
      const int D = e.D, half = D >> 1;
      const int qN = e.Hq * D, kN = e.Hkv * D;
      v0 *= r;
      v1 *= r;
      if (n < qN + kN) {
        const bool isq = n < qN;
        const int nn = isq ? n : n - qN;
        const int head = nn / D, j = (nn - head * D) >> 1;
        const float2 cs = e.rope[(size_t)pos * half + j];
        const float a = v0 * cs.x - v1 * cs.y;  // dim j
        const float c = v1 * cs.x + v0 * cs.y;  // dim j + D/2
        if (isq) {
          size_t base = (((size_t)b * e.Hq + head) * e.Kblk + k) * D;
          st_split<BF>(e.q, e.q_plane, base + j, a);
          st_split<BF>(e.q, e.q_plane, base + j + half, c);
        } else {
          size_t base = (((size_t)b * e.Hkv + head) * e.Lmax + pos) * D;
          st_state<BF>(e.kc, base + j, a);
          st_state<BF>(e.kc, base + j + half, c);
        }
      } else {
        const int nv = n - qN - kN;
        const int head = nv / D, dd = nv - head * D;
        size_t base = (((size_t)b * e.Hkv + head) * D + dd) * e.Lmax + pos;
        st_state<BF>(e.vc, base, v0);
        st_state<BF>(e.vc, base + e.Lmax, v1);
      }
      return 0.f;
    }
    case EPI_RESID: {
      size_t i = (size_t)t * e.ld + n;
      float2 xo = *(const float2*)(e.x + i);
      float x0 = xo.x + v0, x1 = xo.y + v1;
      *(float2*)(e.x + i) = make_float2(x0, x1);
      st_split<BF>(e.xn, e.xn_plane, i, e.gnext[n] * x0);
      st_split<BF>(e.xn, e.xn_plane, i + 1, e.gnext[n + 1] * x1);
      return x0 * x0 + x1 * x1;
    }
    case EPI_SWIGLU: {
      float g = v0 * r, u = v1 * r;
      float s = g / (1.0f + expf(-g));
      st_split<BF>(e.h, e.h_plane, (size_t)t * e.ld + (n >> 1), s * u);
      return 0.f;
    }
    default: {  // EPI_LOGITS
      size_t i = (size_t)t * e.ld + n;
      *(float2*)(e.logits + i) = make_float2(v0 * r, v1 * r);
      return 0.f;
    }
  }
}

struct GemmKArgs {
  const u32x4* W;
  int N, K, KB;
  int S, kchunks, n_fb;
  const uint16_t* in;
  size_t in_plane;
  int ld_in;
  int M, t0;
  int xcd;
  float* part;
  unsigned* counters;
  EpiArgs epi;
};

// NBUF = 1: the workgroup's whole K-slice is one chunk, loaded in one burst
// (tokens to LDS, weights to registers; the MFMAs of k-block kb start as soon
// as its weights land); NBUF = 2: chunks double-buffered.
template <int MT, int NT, int KCB, int NBUF>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmKArgs a) {
  using X = XStage<MT, KCB>;
  __shared__ __attribute__((aligned(16))) uint16_t xs[NBUF][2 * X::PL];
  __shared__ float sq_red[4][X::MP];
  __shared__ float rscale[X::MP];
  __shared__ float rms_red[NBUF == 1 ? 256 : 16 * X::MP];
  __shared__ int is_last;

  int fb, s;
  xcd_unmap(blockIdx.x, a.S, a.xcd, fb, s);
  if (fb >= a.n_fb) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nb0 = (fb * 4 + w) * NT;
  const int kb_split = s * a.kchunks * KCB;
  const uint16_t* in = a.in;
  const int nc = a.kchunks;
  const EpiArgs& e = a.epi;

  floatx4 acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  EpiOps<NT, MT> op;
  u32x4 ra[NBUF][NT][KCB];
  u32x4 rx[2][X::PASSES];

  if constexpr (NBUF == 1) {
    // issue order: block starts, rms partial sums, tokens, then the weight
    // burst; nothing is waited for before the whole burst is in flight
    float rv[RmsPre<X::MP>::RQ];
    epi_block_starts<NT, MT>(e, a.M, a.t0, lane, op);
    rms_issue<X::MP>(e, in, a.M, a.t0, rv);
    load_x<MT, KCB>(rx, in, a.in_plane, a.ld_in, a.M, kb_split * 32);
    load_a<NT, KCB>(ra[0], a.W, a.KB, nb0, a.N, kb_split, lane);
    __builtin_amdgcn_sched_barrier(0);
    rms_finish<X::MP>(e, rv, rms_red, rscale);
    store_x<MT, KCB>(rx, xs[0]);
    lds_barrier();
    compute_chunk<MT, NT, KCB>(acc, ra[0], xs[0], lane);
  } else {
    epi_block_starts<NT, MT>(e, a.M, a.t0, lane, op);
    load_x<MT, KCB>(rx, in, a.in_plane, a.ld_in, a.M, kb_split * 32);
    load_a<NT, KCB>(ra[0], a.W, a.KB, nb0, a.N, kb_split, lane);
    if (e.ssq)
      rms_prologue<X::MP>(e, a.M, a.t0, (float(*)[X::MP])rms_red, rscale);
    else if (threadIdx.x < X::MP)
      rscale[threadIdx.x] = 1.f;
    store_x<MT, KCB>(rx, xs[0]);
    lds_barrier();
    for (int c = 0; c < nc; c += 2) {
      if (c + 1 < nc) {
        load_x<MT, KCB>(rx, in, a.in_plane, a.ld_in, a.M, (kb_split + (c + 1) * KCB) * 32);
        load_a<NT, KCB>(ra[1], a.W, a.KB, nb0, a.N, kb_split + (c + 1) * KCB, lane);
      }
      compute_chunk<MT, NT, KCB>(acc, ra[0], xs[0], lane);
      if (c + 1 < nc) store_x<MT, KCB>(rx, xs[1]);
      lds_barrier();
      if (c + 1 >= nc) break;
      if (c + 2 < nc) {
        load_x<MT, KCB>(rx, in, a.in_plane, a.ld_in, a.M, (kb_split + (c + 2) * KCB) * 32);
        load_a<NT, KCB>(ra[0], a.W, a.KB, nb0, a.N, kb_split + (c + 2) * KCB, lane);
      }
      compute_chunk<MT, NT, KCB>(acc, ra[1], xs[1], lane);
      if (c + 2 < nc) store_x<MT, KCB>(rx, xs[0]);
      lds_barrier();
    }
  }

  if (a.S > 1) {
    // split-K: publish partial fragments, the last workgroup of this feature block reduces
    const size_t frag = (size_t)NT * MT * 64 * 4;
    float* P = a.part + ((size_t)fb * 4 + w) * frag;
    const size_t split_stride = (size_t)a.n_fb * 4 * frag;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        *(floatx4*)(P + (size_t)s * split_stride + ((nt * MT + mt) * 64 + lane) * 4) = acc[nt][mt];
    // every wave's partial stores acknowledged (they sit in this XCD's L2)
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
      if (!a.xcd) __threadfence();  // splits on different XCDs: write back through L2
      unsigned prev = atomicAdd(&a.counters[fb], 1u);
      is_last = (prev == (unsigned)(a.S - 1));
      if (is_last && !a.xcd) __threadfence();
    }
    __syncthreads();
    if (!is_last) return;
  }
  // epilogue operands first, then (split-K) the partials, summed in split
  // order; eight splits' loads are in flight together (indexes clamped, the
  // surplus masked out of the sum, so no branch sits between the loads)
  epi_load<NT, MT>(e, nb0, a.N, a.M, a.t0, lane, op);
  if (a.S > 1) {
    const size_t frag = (size_t)NT * MT * 64 * 4;
    const float* P = a.part + ((size_t)fb * 4 + w) * frag + lane * 4;
    const size_t split_stride = (size_t)a.n_fb * 4 * frag;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < a.S; s0 += 8) {
      floatx4 pv[8][NT][MT];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float* Ps = P + (size_t)min(s0 + j, a.S - 1) * split_stride;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) pv[j][nt][mt] = *(const floatx4*)(Ps + (nt * MT + mt) * 64 * 4);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float m = (s0 + j < a.S) ? 1.f : 0.f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) acc[nt][mt] += pv[j][nt][mt] * m;
      }
    }
    if (threadIdx.x == 0) a.counters[fb] = 0u;
  }

  // epilogue (rscale was filled before the first barrier)
  float sq[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) sq[mt] = 0.f;
  epi_store<NT, MT>(e, acc, op, nb0, a.N, a.M, a.t0, lane, rscale, sq);
  if (e.kind == EPI_RESID) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) sq_red[w][mt * 16 + lane] = v;
    }
    __syncthreads();
    if (threadIdx.x < X::MP && threadIdx.x < a.M) {
      int tl = threadIdx.x;
      float v = ((sq_red[0][tl] + sq_red[1][tl]) + sq_red[2][tl]) + sq_red[3][tl];
      e.ssq_out[(size_t)fb * e.ssq_out_ld + a.t0 + tl] = v;
    }
  }
}

// Wide workgroups for one-burst GEMMs: WV waves, each one 16-feature tile of
// one 512-input K-slice, so that one workgroup per CU covers the launch.  A
// grid of 4-wave workgroups that puts two workgroups on some CUs and one on
// others finishes when the doubled CUs have received twice the bytes
// (measured on a 384-workgroup QKV launch: those workgroups' weights landed
// about 2 us after the others').  The K-slice's token rows are staged
// through registers into LDS, their loads issued before the weights'.
template <int MT, int WV>
__global__ __launch_bounds__(WV * 64) void gemm_wide_kernel(GemmKArgs a) {
  constexpr int KCB = 16, NTH = WV * 64;
  using X = XStage<MT, KCB>;
  using RP = RmsPre<X::MP, GEMM_RMS_MAX_PARTS, NTH>;
  __shared__ __attribute__((aligned(16))) uint16_t xs[2 * X::PL];
  __shared__ float sq_red[WV][X::MP];
  __shared__ float rscale[X::MP];
  __shared__ float rms_red[NTH];
  __shared__ int is_last;

  int fb, s;
  xcd_unmap(blockIdx.x, a.S, a.xcd, fb, s);
  if (fb >= a.n_fb) return;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nb0 = fb * WV + w;
  const int kb_split = s * KCB;
  const EpiArgs& e = a.epi;

  floatx4 acc[1][MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[0][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  EpiOps<1, MT> op;
  u32x4 ra[1][KCB];
  float rv[RP::RQ];
  // issue order: block starts, rms partial sums, token rows, weights; the
  // token rows go to LDS as soon as they land, the weights keep streaming
  using XT = XStage<MT, KCB, NTH>;
  u32x4 rx[2][XT::PASSES];
  epi_block_starts<1, MT>(e, a.M, a.t0, lane, op);
  rms_issue<X::MP, PlainMem, GEMM_RMS_MAX_PARTS, NTH>(e, a.in, a.M, a.t0, rv);
  load_x<MT, KCB, XT::PASSES, PlainMem, NTH>(rx, a.in, a.in_plane, a.ld_in, a.M, kb_split * 32);
  load_a<1, KCB>(ra, a.W, a.KB, nb0, a.N, kb_split, lane);
  __builtin_amdgcn_sched_barrier(0);
  rms_finish<X::MP, GEMM_RMS_MAX_PARTS, NTH>(e, rv, rms_red, rscale);
  store_x<MT, KCB, XT::PASSES, NTH>(rx, xs);
  lds_barrier();
  compute_chunk<MT, 1, KCB>(acc, ra, xs, lane);

  if (a.S > 1) {
    const size_t frag = (size_t)MT * 64 * 4;
    float* P = a.part + ((size_t)fb * WV + w) * frag;
    const size_t split_stride = (size_t)a.n_fb * WV * frag;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) *(floatx4*)(P + (size_t)s * split_stride + (mt * 64 + lane) * 4) = acc[0][mt];
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
      if (!a.xcd) __threadfence();
      unsigned prev = atomicAdd(&a.counters[fb], 1u);
      is_last = (prev == (unsigned)(a.S - 1));
      if (is_last && !a.xcd) __threadfence();
    }
    __syncthreads();
    if (!is_last) return;
  }
  epi_load<1, MT>(e, nb0, a.N, a.M, a.t0, lane, op);
  if (a.S > 1) {
    const size_t frag = (size_t)MT * 64 * 4;
    const float* P = a.part + ((size_t)fb * WV + w) * frag + lane * 4;
    const size_t split_stride = (size_t)a.n_fb * WV * frag;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[0][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    // splits in flight: 64-row tiles keep four (64 registers) so that the
    // 11- and 16-wave workgroups fit their register share without spilling
    constexpr int SB = MT >= 4 ? 4 : 8;
    for (int s0 = 0; s0 < a.S; s0 += SB) {
      floatx4 pv[SB][MT];
#pragma unroll
      for (int j = 0; j < SB; ++j) {
        const float* Ps = P + (size_t)min(s0 + j, a.S - 1) * split_stride;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) pv[j][mt] = *(const floatx4*)(Ps + mt * 64 * 4);
      }
#pragma unroll
      for (int j = 0; j < SB; ++j) {
        const float m = (s0 + j < a.S) ? 1.f : 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[0][mt] += pv[j][mt] * m;
      }
    }
    if (threadIdx.x == 0) a.counters[fb] = 0u;
  }
  float sq[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) sq[mt] = 0.f;
  epi_store<1, MT>(e, acc, op, nb0, a.N, a.M, a.t0, lane, rscale, sq);
  if (e.kind == EPI_RESID) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) sq_red[w][mt * 16 + lane] = v;
    }
    __syncthreads();
    if (threadIdx.x < X::MP && threadIdx.x < a.M) {
      const int tl = threadIdx.x;
      float v = 0.f;
#pragma unroll
      for (int ww = 0; ww < WV; ++ww) v += sq_red[ww][tl];
      e.ssq_out[(size_t)fb * e.ssq_out_ld + a.t0 + tl] = v;
    }
  }
}

GemmPlan gemm_plan_bf16(int M, int N, int K, int xcd) {
  GemmPlan p;
  p.xcd = xcd;
  // up to 128 tokens: one-burst launches over row tiles of at most 64
  // (the weights are streamed once per tile); beyond: double-buffered chunks
  // of 128-row tiles
  int Mc = M <= 128 ? (M < 64 ? M : 64) : 128;
  p.MT = Mc <= 16 ? 1 : Mc <= 32 ? 2 : Mc <= 64 ? 4 : 8;
  const int kb = K / 32;
  if (p.MT <= 4) {
    // one burst per workgroup: the smallest split count whose K-slice (8 or 16
    // k-blocks; 8 for 64-row tiles, whose 16-block token stage would not leave
    // LDS for two workgroups per CU) fits registers and LDS, preferring >= 256
    // workgroups.  Two 16-feature tiles per wave when one tile per wave would
    // need more workgroups than two per CU hold at once (not for 64-row tiles:
    // 340 registers per lane, one wave per SIMD).
    auto burst = [&](int nt, int& n_fb, int& S) {
      n_fb = (N + 64 * nt - 1) / (64 * nt);
      S = 0;
      for (int s = 1; s <= kb; ++s) {
        if (kb % s) continue;
        const int kcb = kb / s;
        if (kcb != 16 && kcb != 8) continue;
        if (p.MT == 4 && kcb != 8) continue;
        if (S == 0) S = s;
        if (n_fb * s >= 256) {
          S = s;
          break;
        }
      }
    };
    int f1, s1, f2, s2;
    burst(1, f1, s1);
    burst(2, f2, s2);
    const bool two = p.MT <= 2 && s2 && kb / s2 == 16 && (!s1 || f1 * s1 > 512);
    if (two || s1) {
      p.NT = two ? 2 : 1;
      p.WV = 4;
      p.bn = 64 * p.NT;
      p.n_fb = two ? f2 : f1;
      p.S = two ? s2 : s1;
      p.KCB = kb / p.S;
      p.kchunks = 1;
      // Wide workgroups when two-tile waves leave the CUs unevenly loaded
      // (grid not a multiple of the 256 CUs) and wide ones cover them exactly
      // once each, cost = bytes through the busiest CU (weights + token rows).
      // Measured on the 1B shapes: gate/up (352 two-tile workgroups -> 256 of
      // 11 waves) 18.2 -> 16.4 us; one-tile grids (QKV 384 -> 256 of 6 waves,
      // down 352 -> 176 of 8) and even grids (LM head 512) got slower.
      auto cost = [&](int grid, int wv, int nt, int kcb) {
        return (double)((grid + 255) / 256) * ((double)wv * nt * kcb * 1024 + (double)Mc * kcb * 32 * 4);
      };
      double best = cost(p.n_fb * p.S, 4, p.NT, p.KCB);
      if (p.MT == 4 && kb % 16 == 0 && N % 16 == 0) {
        // 64-row tiles: the 4-wave plan needs 8-block slices, twice the splits
        // (partial sums ~ splits x N x 64 rows); wide workgroups take 16-block
        // slices, one workgroup per CU, wherever the cost model favours them
        // (on the 1B shapes: all projections except the O projection; gate/up
        // as 256 workgroups of 11 waves, down as 176 of 8).
        for (int wv : {6, 8, 11, 16}) {
          if ((N / 16) % wv) continue;
          const int nfb = N / 16 / wv, S = kb / 16;
          const double c = cost(nfb * S, wv, 1, 16);
          if (c < 0.95 * best) {
            best = c;
            p.WV = wv;
            p.NT = 1;
            p.bn = 16 * wv;
            p.n_fb = nfb;
            p.S = S;
            p.KCB = 16;
          }
        }
      }
      if (p.MT <= 2 && p.NT == 2 && (p.n_fb * p.S) % 256 != 0 && kb % 16 == 0 && N % 16 == 0) {
        for (int wv : {6, 8, 11, 16}) {
          if ((N / 16) % wv) continue;
          const int nfb = N / 16 / wv, S = kb / 16;
          if ((nfb * S) % 256 != 0) continue;
          const double c = cost(nfb * S, wv, 1, 16);
          if (c < 0.95 * best) {
            best = c;
            p.WV = wv;
            p.NT = 1;
            p.bn = 16 * wv;
            p.n_fb = nfb;
            p.S = S;
            p.KCB = 16;
          }
        }
      }
      return p;
    }
  }
  // double-buffered chunks
  p.WV = 4;
  p.NT = p.MT >= 4 ? 2 : 1;
  p.bn = 4 * p.NT * 16;
  p.n_fb = (N + p.bn - 1) / p.bn;
  p.KCB = p.MT == 1 ? 8 : p.MT == 2 ? 4 : p.MT == 4 ? 2 : 1;
  int kch = K / (p.KCB * 32);
  p.S = 1;
  if (p.n_fb < 480) {
    int best = 1;
    for (int s = 1; s <= kch && s <= 16; ++s) {
      if (kch % s) continue;
      best = s;
      if (p.n_fb * s >= 480) break;
    }
    p.S = best;
  }
  p.kchunks = kch / p.S;
  return p;
}

size_t gemm_partials_floats(const GemmPlan& p, int M) {
  (void)M;
  if (p.S <= 1) return 0;
  return (size_t)p.S * p.n_fb * p.WV * p.NT * p.MT * 64 * 4;
}

template <int MT, int WV>
static void launch_wide(const GemmKArgs& a, int n_fb, int S, hipStream_t st) {
  launch_timed(gemm_wide_kernel<MT, WV>, dim3(xcd_grid(n_fb, S, a.xcd)), dim3(WV * 64), st, a);
}

template <int MT>
static void launch_wide_mt(int wv, const GemmKArgs& a, int n_fb, int S, hipStream_t st) {
  switch (wv) {
    case 6: launch_wide<MT, 6>(a, n_fb, S, st); break;
    case 8: launch_wide<MT, 8>(a, n_fb, S, st); break;
    case 11: launch_wide<MT, 11>(a, n_fb, S, st); break;
    default: launch_wide<MT, 16>(a, n_fb, S, st); break;
  }
}

template <int MT, int NT, int KCB, int NBUF>
static void launch_gemm(const GemmKArgs& a, int n_fb, int S, hipStream_t st) {
  launch_timed(gemm_bf16_kernel<MT, NT, KCB, NBUF>, dim3(xcd_grid(n_fb, S, a.xcd)), dim3(256), st, a);
}

void gemm_bf16(const GemmPlan& p, const void* Wpacked, int N, int K, const void* in, size_t in_plane, int ld_in,
               int M, const EpiArgs& epi, float* partials, unsigned* counters, hipStream_t st) {
  const int MP = p.MT * 16;
  for (int t0 = 0; t0 < M; t0 += MP) {
    GemmKArgs a;
    a.W = (const u32x4*)Wpacked;
    a.N = N;
    a.K = K;
    a.KB = K / 32;
    a.S = p.S;
    a.kchunks = p.kchunks;
    a.n_fb = p.n_fb;
    a.in = (const uint16_t*)in + (size_t)t0 * ld_in;
    a.in_plane = in_plane;
    a.ld_in = ld_in;
    a.M = (M - t0) < MP ? (M - t0) : MP;
    a.t0 = t0;
    a.xcd = p.S > 1 ? p.xcd : 0;
    a.part = partials;
    a.counters = counters;
    a.epi = epi;
    if (p.WV != 4) {
      if (p.MT == 1) launch_wide_mt<1>(p.WV, a, p.n_fb, p.S, st);
      else if (p.MT == 2) launch_wide_mt<2>(p.WV, a, p.n_fb, p.S, st);
      else launch_wide_mt<4>(p.WV, a, p.n_fb, p.S, st);
      continue;
    }
    switch (p.MT) {
      case 1:
        if (p.kchunks == 1 && p.KCB == 16 && p.NT == 2) launch_gemm<1, 2, 16, 1>(a, p.n_fb, p.S, st);
        else if (p.kchunks == 1 && p.KCB == 16) launch_gemm<1, 1, 16, 1>(a, p.n_fb, p.S, st);
        else if (p.kchunks == 1 && p.KCB == 8) launch_gemm<1, 1, 8, 1>(a, p.n_fb, p.S, st);
        else launch_gemm<1, 1, 8, 2>(a, p.n_fb, p.S, st);
        break;
      case 2:
        if (p.kchunks == 1 && p.KCB == 16 && p.NT == 2) launch_gemm<2, 2, 16, 1>(a, p.n_fb, p.S, st);
        else if (p.kchunks == 1 && p.KCB == 16) launch_gemm<2, 1, 16, 1>(a, p.n_fb, p.S, st);
        else if (p.kchunks == 1 && p.KCB == 8) launch_gemm<2, 1, 8, 1>(a, p.n_fb, p.S, st);
        else launch_gemm<2, 1, 4, 2>(a, p.n_fb, p.S, st);
        break;
      case 4:
        if (p.kchunks == 1 && p.KCB == 8 && p.NT == 1) launch_gemm<4, 1, 8, 1>(a, p.n_fb, p.S, st);
        else launch_gemm<4, 2, 2, 2>(a, p.n_fb, p.S, st);
        break;
      default: launch_gemm<8, 2, 1, 2>(a, p.n_fb, p.S, st); break;
    }
  }
}

// ---------------- fp32 path (small fp32 models) ----------------
// One thread per (token, output pair); plain fp32 FMAs in k order.
__global__ void gemm_f32_kernel(const float* W, int N, int K, const float* in, int ld_in, int M, EpiArgs e) {
  const int pair = blockIdx.x * blockDim.x + threadIdx.x;
  const int t = blockIdx.y;
  const int n = pair * 2;
  if (n >= N || t >= M) return;
  const float* x = in + (size_t)t * ld_in;
  const float* w0 = W + (size_t)n * K;
  const float* w1 = w0 + K;
  float a0 = 0.f, a1 = 0.f;
  for (int k = 0; k < K; ++k) {
    float xv = x[k];
    a0 = fmaf(xv, w0[k], a0);
    a1 = fmaf(xv, w1[k], a1);
  }
  float r = rms_scale(e, t);
  epi_pair<false>(e, t, n, a0, a1, r);
}

void gemm_f32(const float* W, int N, int K, const float* in, int ld_in, int M, const EpiArgs& epi, hipStream_t st) {
  int pairs = N / 2;
  dim3 grid((pairs + 127) / 128, M);
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(128), 0, st, W, N, K, in, ld_in, M, epi);
}

// ---------------- weight packing ----------------
__global__ void pack_tiles_kernel(const uint16_t* src, const int* rowmap, int N, int K, u32x4* dst) {
  const int KB = K / 32;
  const size_t tiles = (size_t)(N / 16) * KB;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t tile = gid >> 6;
  const int lane = gid & 63;
  if (tile >= tiles) return;
  const int nb = (int)(tile / KB), kb = (int)(tile % KB);
  const int row = rowmap[nb * 16 + (lane & 15)];
  const uint16_t* p = src + (size_t)row * K + kb * 32 + (lane >> 4) * 8;
  u32x4 v;
  v.x = (uint32_t)p[0] | ((uint32_t)p[1] << 16);
  v.y = (uint32_t)p[2] | ((uint32_t)p[3] << 16);
  v.z = (uint32_t)p[4] | ((uint32_t)p[5] << 16);
  v.w = (uint32_t)p[6] | ((uint32_t)p[7] << 16);
  dst[tile * 64 + lane] = v;
}

void pack_bf16_tiles(const uint16_t* src, const int* rowmap, int N, int K, void* dst, hipStream_t st) {
  size_t threads = (size_t)(N / 16) * (K / 32) * 64;
  hipLaunchKernelGGL(pack_tiles_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, src, rowmap, N, K,
                     (u32x4*)dst);
}

__global__ void gather_rows_kernel(const float* src, const int* rowmap, int N, int K, float* dst) {
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= (size_t)N * K) return;
  const int n = (int)(gid / K), k = (int)(gid % K);
  dst[gid] = src[(size_t)rowmap[n] * K + k];
}

void gather_rows_f32(const float* src, const int* rowmap, int N, int K, float* dst, hipStream_t st) {
  size_t total = (size_t)N * K;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, src, rowmap, N, K,
                     dst);
}

}  // namespace ssd
