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
#include <cstdlib>
#include <cstring>

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
  int ft0;  // eight-wave tiles: first 16-feature tile of the launch (its partials and counters count from its first tile)
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

// Tiled GEMM for more than 64 token rows (prefill, batches, guided passes):
// there the weights are worth reusing from registers and LDS rather than
// streaming once per 64-row tile, and from a few hundred rows on the product
// is bound by the matrix cores, not by the weight stream.  Each
// workgroup owns a 128-row x (32 NT)-feature output tile over the whole K
// range and every operand byte it loads feeds many MFMAs.  Four waves in a
// 2 x 2 arrangement, each 64 rows (four 16-row tiles) x 16 NT features; K
// advances in 64-input stages: the stage's token rows (both planes) sit in
// LDS, double-buffered, and each wave's weight fragments (prepacked, one
// 16-byte load per lane each) go straight to registers, the next stage's
// loads in flight while the current stage is multiplied.  All row tiles of a
// feature tile run on one XCD (xcd_grid with the row tiles as the group), so
// its weights come from HBM once and from that XCD's L2 after.  When the
// tiles cannot fill the CUs (few rows, narrow outputs) the K range is split
// over S workgroups of the same XCD; the last of them sums the partials in
// split order and runs the epilogue.
// LDS rows of one stage are unpadded (64 inputs, eight 16-byte chunks); chunk
// c of row r sits at chunk c ^ ((r >> 1) & 7), so that the 16 rows an MFMA
// operand read touches at one logical chunk hit distinct banks in groups of
// 16 and of 32 lanes, and each row's stores stay one 128-byte span
constexpr int TILE_ROWS = 128, TILE_KT = 64, TILE_LD = TILE_KT;
constexpr int TILE_PL = TILE_ROWS * TILE_LD;  // one plane of one stage (bf16)

template <int NT>
struct TileStage {
  u32x4 x[8];         // token rows: 4 rows x 2 planes per thread
  u32x4 w[NT][2];     // weight fragments: NT feature tiles x 2 k-blocks
};

// Buffer loads: a scalar base, 32-bit lane offsets and a scalar offset for
// the stage's K position, the plane and the feature tile.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void* b) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(b), 0, 0x7FFFFFFF, 0x00020000);
}

template <int NT>
__device__ __forceinline__ void tile_load(TileStage<NT>& st, __amdgpu_buffer_rsrc_t xh, __amdgpu_buffer_rsrc_t xl,
                                          const int (&xoff)[4], __amdgpu_buffer_rsrc_t wr, int lane_b, int wtile_b,
                                          int KB, int k0) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    st.x[2 * p] = __builtin_amdgcn_raw_buffer_load_b128(xh, xoff[p], k0 * 2, 0);
    st.x[2 * p + 1] = __builtin_amdgcn_raw_buffer_load_b128(xl, xoff[p], k0 * 2, 0);
  }
  const int kb0 = k0 / 32;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      st.w[nt][kb] = __builtin_amdgcn_raw_buffer_load_b128(wr, lane_b, wtile_b + (nt * KB + kb0 + kb) * 1024, 0);
}

template <int NT>
__device__ __forceinline__ void tile_load_x(TileStage<NT>& st, __amdgpu_buffer_rsrc_t xh, __amdgpu_buffer_rsrc_t xl,
                                            const int (&xoff)[4], int k0) {
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    st.x[2 * p] = __builtin_amdgcn_raw_buffer_load_b128(xh, xoff[p], k0 * 2, 0);
    st.x[2 * p + 1] = __builtin_amdgcn_raw_buffer_load_b128(xl, xoff[p], k0 * 2, 0);
  }
}

template <int NT>
__device__ __forceinline__ void tile_load_w(TileStage<NT>& st, __amdgpu_buffer_rsrc_t wr, int lane_b, int wtile_b,
                                            int KB, int k0) {
  const int kb0 = k0 / 32;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      st.w[nt][kb] = __builtin_amdgcn_raw_buffer_load_b128(wr, lane_b, wtile_b + (nt * KB + kb0 + kb) * 1024, 0);
}

template <int NT>
__device__ __forceinline__ void tile_store_x(const TileStage<NT>& st, uint16_t* xs, int tid) {
  const int cg = tid & 7, rr = tid >> 3;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int r = rr + 32 * p;
    const int pc = cg ^ ((r >> 1) & 7);
    *(u32x4*)(xs + r * TILE_LD + pc * 8) = st.x[2 * p];
    *(u32x4*)(xs + TILE_PL + r * TILE_LD + pc * 8) = st.x[2 * p + 1];
  }
}

template <int NT>
__device__ __forceinline__ void tile_mma(floatx4 (&acc)[NT][4], const TileStage<NT>& st, const uint16_t* xs, int wm,
                                         int lane) {
  const int row = wm * 64 + (lane & 15);
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    bf16x8 bhi[4], blo[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      // rows row + 16 mt share (row >> 1) & 7 = ((lane & 15) >> 1)
      const uint16_t* p = xs + (row + mt * 16) * TILE_LD + (((kb * 4 + (lane >> 4)) ^ ((lane & 15) >> 1)) * 8);
      bhi[mt] = __builtin_bit_cast(bf16x8, *(const u32x4*)p);
      blo[mt] = __builtin_bit_cast(bf16x8, *(const u32x4*)(p + TILE_PL));
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const bf16x8 w = __builtin_bit_cast(bf16x8, st.w[nt][kb]);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, bhi[mt], acc[nt][mt], 0, 0, 0);
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, blo[mt], acc[nt][mt], 0, 0, 0);
      }
    }
  }
}

// DEPTH 2: two register stages, loads one stage ahead; DEPTH 4: four
// register stages, loads three stages ahead (64-feature tiles only, which
// still fit two workgroups per CU with them)
template <int NT, int DEPTH>
__global__ __launch_bounds__(256, 2) void gemm_tile_kernel(GemmKArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][2 * TILE_PL];
  __shared__ float rscale[TILE_ROWS];
  __shared__ float sq_red[2][TILE_ROWS];

  __shared__ int is_last;
  const int m_tiles = (a.M + TILE_ROWS - 1) / TILE_ROWS;
  int fb, member;
  xcd_unmap(blockIdx.x, m_tiles * a.S, a.xcd, fb, member);
  if (fb >= a.n_fb) return;
  const int mtile = member / a.S, split = member - mtile * a.S;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: scalar addressing
  const int wm = w & 1, wn = w >> 1;
  const int r0 = mtile * TILE_ROWS;                 // first row of the tile
  const int nb0 = fb * 2 * NT + wn * NT;            // first 16-feature tile of this wave
  const int t0w = a.t0 + r0 + wm * 64;              // first row of this wave (absolute)
  const int Mw = a.M - r0 - wm * 64 < 64 ? a.M - r0 - wm * 64 : 64;  // rows of this wave (<= 0: none)
  const int Mt = a.M - r0 < TILE_ROWS ? a.M - r0 : TILE_ROWS;
  const EpiArgs& e = a.epi;
  const int nst = a.K / TILE_KT / a.S, st0 = split * nst;  // this split's stages (a multiple of DEPTH)

  floatx4 acc[NT][4];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) acc[nt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // lane offsets of the token rows this thread copies (rows past M repeat
  // row M - 1; their results are never stored) and of its weight fragments
  const __amdgpu_buffer_rsrc_t xh = tile_rsrc(a.in), xl = tile_rsrc(a.in + a.in_plane), wr = tile_rsrc(a.W);
  int xoff[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int r = r0 + (tid >> 3) + 32 * p;
    xoff[p] = ((r < a.M ? r : a.M - 1) * a.ld_in + (tid & 7) * 8) * 2;
  }
  const int lane_b = lane * 16, wtile_b = nb0 * a.KB * 1024;
  auto load = [&](TileStage<NT>& st, int stage) {
    tile_load<NT>(st, xh, xl, xoff, wr, lane_b, wtile_b, a.KB, (st0 + stage) * TILE_KT);
  };
  auto load_x = [&](TileStage<NT>& st, int stage) { tile_load_x<NT>(st, xh, xl, xoff, (st0 + stage) * TILE_KT); };
  auto load_w = [&](TileStage<NT>& st, int stage) {
    tile_load_w<NT>(st, wr, lane_b, wtile_b, a.KB, (st0 + stage) * TILE_KT);
  };
  // 1/rms of the tile's rows (the LDS of stage buffer 1 serves as the
  // reduction scratch; it is written only after the next barrier)
  auto rms = [&]() {
    if (e.ssq)
      rms_prologue<TILE_ROWS>(e, Mt, a.t0 + r0, (float(*)[TILE_ROWS])(void*)xs[1], rscale);
    else if (tid < TILE_ROWS)
      rscale[tid] = 1.f;
  };
  // DEPTH stages per trip, so that the register stages have fixed names and
  // the loop body has no branch (a branch makes the compiler move the
  // accumulators between register files every trip); stage c sits in LDS
  // buffer c % 2
  if constexpr (DEPTH == 3) {
    // weights two stages ahead in three register slots (w0..w2), token rows
    // one stage ahead (xr); a trip runs three stages, so the LDS buffer of
    // its first stage alternates between trips
    TileStage<NT> w0, w1, w2, xr;
    load(w0, 0);
    load_w(w1, 1);
    rms();
    tile_store_x<NT>(w0, xs[0], tid);
    lds_barrier();
    int c = 0;
    uint16_t* xa = xs[0];  // buffer of stage c
    uint16_t* xb = xs[1];
    for (; c + 4 < nst; c += 3) {
      load_x(xr, c + 1);
      load_w(w2, c + 2);
      tile_mma<NT>(acc, w0, xa, wm, lane);
      tile_store_x<NT>(xr, xb, tid);
      lds_barrier();
      load_x(xr, c + 2);
      load_w(w0, c + 3);
      tile_mma<NT>(acc, w1, xb, wm, lane);
      tile_store_x<NT>(xr, xa, tid);
      lds_barrier();
      load_x(xr, c + 3);
      load_w(w1, c + 4);
      tile_mma<NT>(acc, w2, xa, wm, lane);
      tile_store_x<NT>(xr, xb, tid);
      lds_barrier();
      uint16_t* t = xa;
      xa = xb;
      xb = t;
    }
    // 2, 3 or 4 stages left: w0 holds stage c (its rows in xa), w1 stage c + 1
    const int left = nst - c;
    load_x(xr, c + 1);
    if (left >= 3) load_w(w2, c + 2);
    tile_mma<NT>(acc, w0, xa, wm, lane);
    tile_store_x<NT>(xr, xb, tid);
    lds_barrier();
    if (left >= 3) {
      load_x(xr, c + 2);
      if (left == 4) load_w(w0, c + 3);
    }
    tile_mma<NT>(acc, w1, xb, wm, lane);
    if (left >= 3) {
      tile_store_x<NT>(xr, xa, tid);
      lds_barrier();
      if (left == 4) load_x(xr, c + 3);
      tile_mma<NT>(acc, w2, xa, wm, lane);
      if (left == 4) {
        tile_store_x<NT>(xr, xb, tid);
        lds_barrier();
        tile_mma<NT>(acc, w0, xb, wm, lane);
      }
    }
  } else if constexpr (DEPTH == 2) {
    TileStage<NT> s0, s1;
    load(s0, 0);
    rms();
    tile_store_x<NT>(s0, xs[0], tid);
    lds_barrier();
    int c = 0;
    for (; c + 2 < nst; c += 2) {
      load(s1, c + 1);
      tile_mma<NT>(acc, s0, xs[0], wm, lane);
      tile_store_x<NT>(s1, xs[1], tid);
      lds_barrier();
      load(s0, c + 2);
      tile_mma<NT>(acc, s1, xs[1], wm, lane);
      tile_store_x<NT>(s0, xs[0], tid);
      lds_barrier();
    }
    load(s1, c + 1);
    tile_mma<NT>(acc, s0, xs[0], wm, lane);
    tile_store_x<NT>(s1, xs[1], tid);
    lds_barrier();
    tile_mma<NT>(acc, s1, xs[1], wm, lane);
  } else {
    TileStage<NT> s0, s1, s2, s3;
    load(s0, 0);
    load(s1, 1);
    load(s2, 2);
    rms();
    tile_store_x<NT>(s0, xs[0], tid);
    lds_barrier();
    int c = 0;
    for (; c + 4 < nst; c += 4) {
      load(s3, c + 3);
      tile_mma<NT>(acc, s0, xs[0], wm, lane);
      tile_store_x<NT>(s1, xs[1], tid);
      lds_barrier();
      load(s0, c + 4);
      tile_mma<NT>(acc, s1, xs[1], wm, lane);
      tile_store_x<NT>(s2, xs[0], tid);
      lds_barrier();
      load(s1, c + 5);
      tile_mma<NT>(acc, s2, xs[0], wm, lane);
      tile_store_x<NT>(s3, xs[1], tid);
      lds_barrier();
      load(s2, c + 6);
      tile_mma<NT>(acc, s3, xs[1], wm, lane);
      tile_store_x<NT>(s0, xs[0], tid);
      lds_barrier();
    }
    load(s3, c + 3);
    tile_mma<NT>(acc, s0, xs[0], wm, lane);
    tile_store_x<NT>(s1, xs[1], tid);
    lds_barrier();
    tile_mma<NT>(acc, s1, xs[1], wm, lane);
    tile_store_x<NT>(s2, xs[0], tid);
    lds_barrier();
    tile_mma<NT>(acc, s2, xs[0], wm, lane);
    tile_store_x<NT>(s3, xs[1], tid);
    lds_barrier();
    tile_mma<NT>(acc, s3, xs[1], wm, lane);
  }

  if (a.S > 1) {
    // split-K: publish this split's fragments; the last arrival of the tile
    // sums all splits in split order (deterministic)
    const int grp = fb * m_tiles + mtile;
    constexpr int FRAG = NT * 4 * 64 * 4;  // floats per wave
    float* P = a.part + ((size_t)grp * a.S * 4 + w) * FRAG + lane * 4;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) *(floatx4*)(P + (size_t)split * 4 * FRAG + (nt * 4 + mt) * 256) = acc[nt][mt];
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
      if (!a.xcd) __threadfence();  // splits on different XCDs: write back through L2
      const unsigned prev = atomicAdd(&a.counters[grp], 1u);
      is_last = prev == (unsigned)(a.S - 1);
      if (is_last && !a.xcd) __threadfence();
    }
    __syncthreads();
    if (!is_last) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) acc[nt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.S; ++sp) {
      floatx4 v[NT][4];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) v[nt][mt] = *(const floatx4*)(P + (size_t)sp * 4 * FRAG + (nt * 4 + mt) * 256);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[nt][mt] += v[nt][mt];
    }
    if (tid == 0) a.counters[grp] = 0u;
  }

  float sq[4] = {0.f, 0.f, 0.f, 0.f};
  if (NT == 2 && e.kind == EPI_RESID) {
    // the new residual x stored in place (16 bytes a lane); both planes of
    // g * x (8 bytes a lane and plane) go through the wave's NT x 4 KiB of the
    // stage buffers and come back as 16 bytes of one row a lane: NT x 32
    // contiguous bytes per row and plane (64-feature tiles only: with 128
    // features the registers this takes spill inside the K loop)
    __syncthreads();  // every wave is done with the stage buffers
    if (Mw > 0) {
      EpiOps<NT, 4> op;
      epi_load<NT, 4>(e, nb0, a.N, Mw, t0w, lane, op);
      constexpr int RL = NT * 16;  // features of a wave row
      uint16_t* stg = &xs[0][0] + w * (2 * 64 * RL);  // [plane][64 rows][RL]
      const int nq = 4 * (lane >> 4);
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = mt * 16 + (lane & 15);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const floatx4 v = acc[nt][mt];
          const float4 xo = op.a[nt][mt], g = op.g[nt];
          const float4 xv = make_float4(xo.x + v[0], xo.y + v[1], xo.z + v[2], xo.w + v[3]);
          if (row < Mw) *(float4*)(e.x + (size_t)(t0w + row) * e.ld + (nb0 + nt) * 16 + nq) = xv;
          uint32_t h0, l0, h1, l1;
          split2(g.x * xv.x, g.y * xv.y, h0, l0);
          split2(g.z * xv.z, g.w * xv.w, h1, l1);
          *(uint2*)(stg + row * RL + nt * 16 + nq) = make_uint2(h0, h1);
          *(uint2*)(stg + 64 * RL + row * RL + nt * 16 + nq) = make_uint2(l0, l1);
          sq[mt] += (xv.x * xv.x + xv.y * xv.y) + (xv.z * xv.z + xv.w * xv.w);
        }
      }
      asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: its reads see all its lanes' writes
      uint16_t* xn = (uint16_t*)e.xn;
      constexpr int CH = RL / 8, RPI = 64 / CH;  // 16-byte chunks per row, rows per instruction
      const int c = lane % CH;
#pragma unroll
      for (int pl = 0; pl < 2; ++pl)
#pragma unroll
        for (int k = 0; k < 64 / RPI; ++k) {
          const int row = k * RPI + lane / CH;
          const uint4 v = *(const uint4*)(stg + pl * 64 * RL + row * RL + c * 8);
          if (row < Mw) *(uint4*)(xn + (pl ? e.xn_plane : 0) + (size_t)(t0w + row) * e.ld + nb0 * 16 + c * 8) = v;
        }
    }
  } else if (Mw > 0) {
    EpiOps<NT, 4> op;
    epi_block_starts<NT, 4>(e, Mw, t0w, lane, op);
    epi_load<NT, 4>(e, nb0, a.N, Mw, t0w, lane, op);
    epi_store<NT, 4>(e, acc, op, nb0, a.N, Mw, t0w, lane, rscale + wm * 64, sq);
  }
  if (e.kind == EPI_RESID) {
    // per-row sums of x^2 over this tile's features: lanes of one row, then
    // the two waves of one row half, in a fixed order
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) sq_red[wn][wm * 64 + mt * 16 + lane] = v;
    }
    __syncthreads();
    if (tid < Mt) e.ssq_out[(size_t)fb * e.ssq_out_ld + a.t0 + r0 + tid] = sq_red[0][tid] + sq_red[1][tid];
  }
}

// ---------------- wide tiles with both operands through an LDS DMA ring ----------------
// Eight waves (two per SIMD, one workgroup per CU) own a 128-row x 256-feature
// output tile: 2 (rows) x 4 (features) waves of 64 x 64, the wave tile of
// gemm_tile_kernel<4, 3>.  A 64-input stage -- the token rows of both planes
// (32 KiB) and the 32 packed 1 KiB weight tiles of the 256 features (32 KiB)
// -- comes by LDS DMA into a ring of two stages, the next stage's copies in
// flight while the current one is multiplied; every operand byte crosses the
// L2 once per workgroup (with the 128 x 128 tiles the token rows crossed it
// once per 128 features and each weight fragment once per wave that uses
// it).  A token DMA instruction fills eight rows x 128 bytes (whole cache
// lines), its lanes choosing the global chunk so that LDS holds the rows in
// the swizzled layout the operand reads expect (chunk c of row r at c ^ ((r
// >> 1) & 7)); a weight tile lands in its stored lane order, so both operand
// reads are one conflict-free ds_read_b128 per fragment.  The reads are
// issued as separate instructions with their own waits, so that the
// compiler does not make them wait for every LDS DMA copy in flight.
// A narrower variant (NT = 3: waves of 64 x 48, tiles of 128 x 192, 24 weight
// tiles a stage in the same ring) fills grids that the 256-feature tiles
// leave part empty.
constexpr int T8_STAGES = 2, T8_THREADS = 512;
constexpr int T8_STAGE_BYTES = 2 * TILE_PL * 2 + 32 * 1024;  // one stage: both token planes, then up to 32 weight tiles

// the eight token operand fragments of one k-block at addr: [mt * 2 + plane],
// row tiles 16 rows (2 KiB) apart, the planes TILE_PL elements apart
__device__ __forceinline__ void ds_read_tiles2(u32x4 (&x)[8], uint32_t addr) {
  constexpr int PL = TILE_PL * 2, RT = 16 * TILE_LD * 2;
  x[0] = ds_read16_at<0>(addr);
  x[1] = ds_read16_at<PL>(addr);
  x[2] = ds_read16_at<RT>(addr);
  x[3] = ds_read16_at<PL + RT>(addr);
  x[4] = ds_read16_at<2 * RT>(addr);
  x[5] = ds_read16_at<PL + 2 * RT>(addr);
  x[6] = ds_read16_at<3 * RT>(addr);
  x[7] = ds_read16_at<PL + 3 * RT>(addr);
}

// K loop of one tile segment: stages st0 .. st0 + nst - 1 of the 128 token
// rows from r0 against the 64 NT features from 16-feature tile ft, summed
// into acc.  pro() runs once the first stage's copies are in flight (the
// tile's 1/rms, whose LDS scratch is the ring's second buffer); on return
// every wave is past the last stage's barrier, so the buffer of stage nst is
// free.
template <int NT, class Pro>
__device__ __forceinline__ void t8_kloop(const GemmKArgs& a, int ft, int r0, int st0, int nst, uint16_t* xs,
                                         floatx4 (&acc)[NT][4], Pro&& pro) {
  static_assert(NT == 3 || NT == 4, "waves of 48 or 64 features");
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int wm = w & 1, wn = w >> 1;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) acc[nt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  const __amdgpu_buffer_rsrc_t xh = tile_rsrc(a.in), xl = tile_rsrc(a.in + a.in_plane), wr = tile_rsrc(a.W);
  // token DMA: 32 instructions a stage (2 planes x 16 blocks of 8 rows), four
  // per wave; lane l of block rb takes row rb * 8 + l / 8 and stored chunk
  // l % 8, i.e. the logical chunk (l % 8) ^ ((row >> 1) & 7) (rows past M
  // repeat row M - 1; their results are never stored)
  int xoff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int i = w * 4 + j, rb = i & 15;
    const int row = rb * 8 + (lane >> 3);
    const int r = r0 + row;
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    xoff[j] = ((r < a.M ? r : a.M - 1) * a.ld_in + c * 8) * 2;
  }
  auto issue_x = [&](int stage) {
    uint16_t* dst = xs + (size_t)(stage % T8_STAGES) * (T8_STAGE_BYTES / 2);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int i = w * 4 + j, pl = i >> 4, rb = i & 15;
      dma16(pl ? xl : xh, dst + pl * TILE_PL + rb * 512, xoff[j], (st0 + stage) * TILE_KT * 2);
    }
    // the stage's 8 NT weight tiles (4 NT feature tiles x 2 k-blocks), NT per wave
    const int kb0 = (st0 + stage) * TILE_KT / 32;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int i = w * NT + j, f = i >> 1, kb = i & 1;
      dma16(wr, dst + 2 * TILE_PL + i * 512, lane * 16, ((ft + f) * a.KB + kb0 + kb) * 1024);
    }
  };
  // operand reads: row wm * 64 + lane % 16 (+ 16 mt), logical chunk kb * 4 +
  // lane / 16 stored at that ^ ((row >> 1) & 7), which no mt changes
  const uint32_t xs0 = lds_addr(xs);
  uint32_t xrd[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
    xrd[kb] = xs0 + (uint32_t)(((wm * 64 + (lane & 15)) * TILE_LD +
                                (((kb * 4 + (lane >> 4)) ^ ((lane & 15) >> 1)) * 8)) * 2);
  // weight tile (f, kb) of the stage sits at (2 f + kb) KiB after its token
  // planes; this wave's feature tiles are f = NT wn .. NT wn + NT - 1
  const uint32_t wrd = xs0 + (uint32_t)(2 * TILE_PL * 2 + wn * NT * 2048 + lane * 16);
  auto mma = [&](int stage) {
    const uint32_t so = (uint32_t)((stage % T8_STAGES) * T8_STAGE_BYTES);
    u32x4 x0[8], x1[8], b0[NT], b1[NT];  // token [mt * 2 + plane] and weight [nt] fragments of k-blocks 0 and 1
    ds_read_tiles2(x0, xrd[0] + so);
    b0[0] = ds_read16_at<0>(wrd + so);
    b0[1] = ds_read16_at<2048>(wrd + so);
    b0[2] = ds_read16_at<4096>(wrd + so);
    if constexpr (NT == 4) b0[NT - 1] = ds_read16_at<6144>(wrd + so);
    ds_read_tiles2(x1, xrd[1] + so);
    b1[0] = ds_read16_at<1024>(wrd + so);
    b1[1] = ds_read16_at<3072>(wrd + so);
    b1[2] = ds_read16_at<5120>(wrd + so);
    if constexpr (NT == 4) b1[NT - 1] = ds_read16_at<7168>(wrd + so);
    lgkm_wait<8 + NT>(x0);  // k-block 0's reads done, k-block 1's (8 + NT) may be outstanding
    lgkm_wait<8 + NT>(b0);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const bf16x8 wf = __builtin_bit_cast(bf16x8, b0[nt]);
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, __builtin_bit_cast(bf16x8, x0[mt * 2]), acc[nt][mt], 0, 0, 0);
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, __builtin_bit_cast(bf16x8, x0[mt * 2 + 1]), acc[nt][mt], 0, 0, 0);
      }
    __builtin_amdgcn_sched_barrier(0);  // the first k-block's MFMAs stay above the second wait
    lgkm_wait<0>(x1);
    lgkm_wait<0>(b1);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const bf16x8 wf = __builtin_bit_cast(bf16x8, b1[nt]);
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, __builtin_bit_cast(bf16x8, x1[mt * 2]), acc[nt][mt], 0, 0, 0);
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, __builtin_bit_cast(bf16x8, x1[mt * 2 + 1]), acc[nt][mt], 0, 0, 0);
      }
  };

  issue_x(0);
  pro();
  // stage c: this wave's copies of stage c are done (none are issued after
  // them yet), the barrier publishes everyone's copies and tells that every
  // wave is done with stage c - 1, whose ring buffer then takes stage c + 1
  for (int c = 0; c < nst; ++c) {
    wait_vmcnt<0>();
    dma_barrier();
    if (c + 1 < nst) issue_x(c + 1);
    mma(c);
  }
}

// x * sigmoid(x) from the hardware exp2 and reciprocal (each within about
// one ulp; the limits 0 and x hold for large |x|)
__device__ __forceinline__ float silu_hw(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -1.44269504088896341f));
}

// Epilogue of the tile (fb, rows r0 ..) from its sums; stg: a free ring
// buffer (64 KiB).  Every thread of the workgroup calls it (one barrier for
// the residual's row sums).
template <int NT>
__device__ __forceinline__ void t8_epilogue(const GemmKArgs& a, int fb, int ft, int r0, const floatx4 (&acc)[NT][4],
                                            const float* rscale, float (*sq_red)[TILE_ROWS], uint16_t* stg_all) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w & 1, wn = w >> 1;
  const int nb0 = ft + wn * NT;  // first 16-feature tile of this wave
  const int t0w = a.t0 + r0 + wm * 64;
  const int Mw = a.M - r0 - wm * 64 < 64 ? a.M - r0 - wm * 64 : 64;
  const int Mt = a.M - r0 < TILE_ROWS ? a.M - r0 : TILE_ROWS;
  const EpiArgs& e = a.epi;
  float sq[4] = {0.f, 0.f, 0.f, 0.f};
  if (e.kind == EPI_SWIGLU) {
    // a lane's four features of one fragment are two gate/up pairs, i.e. two
    // adjacent outputs (4 bytes a plane): the wave's 64 x 32 outputs go
    // through its own 8 KiB of the free ring buffer and come back as 16
    // bytes of one row a lane, stored as 64 contiguous bytes per row and plane
    if (Mw > 0) {
      uint16_t* stg = stg_all + w * 4096;  // [plane][64 rows][32]
      const int q = lane >> 4;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = mt * 16 + (lane & 15);
        const float r = rscale[wm * 64 + row];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const floatx4 v = acc[nt][mt];
          const float g0 = v[0] * r, u0 = v[1] * r, g1 = v[2] * r, u1 = v[3] * r;
          uint32_t hi, lo;
          split2(silu_hw(g0) * u0, silu_hw(g1) * u1, hi, lo);
          *(uint32_t*)(stg + row * 32 + nt * 8 + 2 * q) = hi;
          *(uint32_t*)(stg + 2048 + row * 32 + nt * 8 + 2 * q) = lo;
        }
      }
      asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: its reads see all its lanes' writes
      uint16_t* h = (uint16_t*)e.h;
      const int c = lane & 3;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int row = k * 16 + (lane >> 2);
        const uint4 hi = *(const uint4*)(stg + row * 32 + c * 8);
        const uint4 lo = *(const uint4*)(stg + 2048 + row * 32 + c * 8);
        if (row < Mw && c < NT) {  // a wave's 8 NT outputs of a row are NT chunks
          const size_t i = (size_t)(t0w + row) * e.ld + nb0 * 8 + c * 8;
          *(uint4*)(h + i) = hi;
          *(uint4*)(h + e.h_plane + i) = lo;
        }
      }
    }
  } else if (e.kind == EPI_RESID) {
    // the new residual x stored in place (16 bytes a lane); the planes of
    // g * x (8 bytes a lane and plane) go through the wave's 8 KiB of the
    // free ring buffer one plane at a time and come back as 16 bytes of one
    // row a lane: 128 contiguous bytes per row and plane
    if (Mw > 0) {
      EpiOps<NT, 4> op;
      epi_load<NT, 4>(e, nb0, a.N, Mw, t0w, lane, op);
      uint16_t* stg = stg_all + w * 4096;  // [64 rows][64 features], one plane
      const int nq = 4 * (lane >> 4);
      uint2 lo[NT][4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = mt * 16 + (lane & 15);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const floatx4 v = acc[nt][mt];
          const float4 xo = op.a[nt][mt], g = op.g[nt];
          const float4 xv = make_float4(xo.x + v[0], xo.y + v[1], xo.z + v[2], xo.w + v[3]);
          if (row < Mw) *(float4*)(e.x + (size_t)(t0w + row) * e.ld + (nb0 + nt) * 16 + nq) = xv;
          uint32_t h0, l0, h1, l1;
          split2(g.x * xv.x, g.y * xv.y, h0, l0);
          split2(g.z * xv.z, g.w * xv.w, h1, l1);
          *(uint2*)(stg + row * 64 + nt * 16 + nq) = make_uint2(h0, h1);
          lo[nt][mt] = make_uint2(l0, l1);
          sq[mt] += (xv.x * xv.x + xv.y * xv.y) + (xv.z * xv.z + xv.w * xv.w);
        }
      }
      uint16_t* xn = (uint16_t*)e.xn;
      const int c = lane & 7;
#pragma unroll
      for (int pl = 0; pl < 2; ++pl) {
        if (pl) {
#pragma unroll
          for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) *(uint2*)(stg + (mt * 16 + (lane & 15)) * 64 + nt * 16 + nq) = lo[nt][mt];
        }
        asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: its reads see all its lanes' writes
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int row = k * 8 + (lane >> 3);
          const uint4 v = *(const uint4*)(stg + row * 64 + c * 8);
          if (row < Mw && c < 2 * NT)
            *(uint4*)(xn + (pl ? e.xn_plane : 0) + (size_t)(t0w + row) * e.ld + nb0 * 16 + c * 8) = v;
        }
        asm volatile("" ::: "memory");  // the lo plane's writes stay behind the hi plane's reads
      }
    }
  } else if (NT == 4 && e.kind == EPI_QKV && nb0 * 16 < e.Hq * e.D && (e.D & 63) == 0) {
    // query features (a wave's 64 features lie in one head: rotary pairs j0 ..
    // j0 + 31 and their partners j0 + D/2 ..): the rotated values, 4 bytes a
    // lane and plane before, go through the wave's 8 KiB of the free ring
    // buffer one plane at a time, [64 tokens][dims j0 .. j0 + 31, then
    // j0 + D/2 ..], and come back as the 8 dims of one tiled-q lane chunk
    // (16 bytes) a lane
    if (Mw > 0) {
      EpiOps<NT, 4> op;
      epi_block_starts<NT, 4>(e, Mw, t0w, lane, op);
      epi_load<NT, 4>(e, nb0, a.N, Mw, t0w, lane, op);
      const int D = e.D, half = D >> 1;
      const int n0 = nb0 * 16, head = n0 / D, j0 = (n0 - head * D) >> 1;
      const int g = e.Hq / e.Hkv, hkv = head / g, hg = head - hkv * g;
      uint16_t* stg = stg_all + w * 4096;
      const int nq = 4 * (lane >> 4);
      uint2 lo[NT][4];  // lo planes of (j, j + 1) and (j + D/2, j + 1 + D/2), for the second pass
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int row = mt * 16 + (lane & 15);
        const float r = rscale[wm * 64 + row];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const floatx4 v = acc[nt][mt];
          const float4 cs = op.a[nt][mt];
          const float x0 = v[0] * r, y0 = v[1] * r, x1 = v[2] * r, y1 = v[3] * r;
          const float a0 = x0 * cs.x - y0 * cs.y, c0 = y0 * cs.x + x0 * cs.y;
          const float a1 = x1 * cs.z - y1 * cs.w, c1 = y1 * cs.z + x1 * cs.w;
          uint32_t h0, l0, h1, l1;
          split2(a0, a1, h0, l0);
          split2(c0, c1, h1, l1);
          const int jj = nt * 8 + nq / 2;  // pair offset from j0 (even)
          *(uint32_t*)(stg + row * 64 + jj) = h0;
          *(uint32_t*)(stg + row * 64 + 32 + jj) = h1;
          lo[nt][mt] = make_uint2(l0, l1);
        }
      }
      uint16_t* qb = (uint16_t*)e.q;
      const int c = lane & 7;
      const int col = c < 4 ? j0 + c * 8 : j0 + half + (c - 4) * 8;
#pragma unroll
      for (int pl = 0; pl < 2; ++pl) {
        if (pl) {
#pragma unroll
          for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
              const int row = mt * 16 + (lane & 15), jj = nt * 8 + nq / 2;
              *(uint32_t*)(stg + row * 64 + jj) = lo[nt][mt].x;
              *(uint32_t*)(stg + row * 64 + 32 + jj) = lo[nt][mt].y;
            }
        }
        asm volatile("" ::: "memory");  // a wave's LDS accesses run in order: its reads see all its lanes' writes
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int row = k * 8 + (lane >> 3);
          const uint4 v = *(const uint4*)(stg + row * 64 + c * 8);
          if (row < Mw) {
            const int t = t0w + row, b = t / e.Kblk, kk = t - b * e.Kblk;
            const size_t base = ((size_t)b * e.Hkv + hkv) * (size_t)e.qrows_pad * D;
            *(uint4*)(qb + (pl ? e.q_plane : 0) + base + tile16x32_index(hg * e.Kblk + kk, col, D)) = v;
          }
        }
        asm volatile("" ::: "memory");  // the lo plane's writes stay behind the hi plane's reads
      }
    }
  } else if (Mw > 0) {
    EpiOps<NT, 4> op;
    epi_block_starts<NT, 4>(e, Mw, t0w, lane, op);
    epi_load<NT, 4>(e, nb0, a.N, Mw, t0w, lane, op);
    epi_store<NT, 4>(e, acc, op, nb0, a.N, Mw, t0w, lane, rscale + wm * 64, sq);
  }
  if (e.kind == EPI_RESID) {
    // per-row sums of x^2 over this tile's features: lanes of one row, then
    // the four waves of one row half, in a fixed order
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) sq_red[wn][wm * 64 + mt * 16 + lane] = v;
    }
    __syncthreads();
    if (tid < Mt)
      e.ssq_out[(size_t)fb * e.ssq_out_ld + a.t0 + r0 + tid] =
          ((sq_red[0][tid] + sq_red[1][tid]) + sq_red[2][tid]) + sq_red[3][tid];
  }
}

// the tile's 1/rms of its rows (1 without a norm), scratch: 8 KiB of LDS
__device__ __forceinline__ void t8_rms(const GemmKArgs& a, int r0, float* scratch, float* rscale) {
  const int Mt = a.M - r0 < TILE_ROWS ? a.M - r0 : TILE_ROWS;
  if (a.epi.ssq)
    rms_prologue<TILE_ROWS, T8_THREADS>(a.epi, Mt, a.t0 + r0, (float(*)[TILE_ROWS])(void*)scratch, rscale);
  else if (threadIdx.x < TILE_ROWS)
    rscale[threadIdx.x] = 1.f;
}

// One workgroup per output tile and K split (grid of xcd_grid(n_fb,
// m_tiles * S)): the splits' sums meet in the last arrival.  Feature block fb
// of the launch covers the 4 NT 16-feature tiles from a.ft0 + 4 NT fb; its
// per-row x^2 part (residual epilogue) is number ft / (4 NT), which counts
// the blocks of the whole projection when every launch of it has one width.
template <int NT>
__global__ __launch_bounds__(T8_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_tile8_kernel(GemmKArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[T8_STAGES * T8_STAGE_BYTES / 2];
  __shared__ float rscale[TILE_ROWS];
  __shared__ float sq_red[4][TILE_ROWS];
  __shared__ int is_last;
  const int m_tiles = (a.M + TILE_ROWS - 1) / TILE_ROWS;
  int fb, member;
  xcd_unmap(blockIdx.x, m_tiles * a.S, a.xcd, fb, member);
  if (fb >= a.n_fb) return;
  const int mtile = member / a.S, split = member - mtile * a.S;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int r0 = mtile * TILE_ROWS;
  const int nst = a.K / TILE_KT / a.S;

  const int ft = a.ft0 + fb * 4 * NT;  // the tile's first 16-feature tile
  floatx4 acc[NT][4];
  t8_kloop<NT>(a, ft, r0, split * nst, nst, xs, acc,
               [&] { t8_rms(a, r0, (float*)(void*)(xs + T8_STAGE_BYTES / 2), rscale); });

  if (a.S > 1) {
    // split-K: publish this split's fragments; the last arrival of the tile
    // sums all splits in split order (deterministic)
    const int grp = fb * m_tiles + mtile;
    constexpr int FRAG = NT * 4 * 64 * 4;  // floats per wave
    float* P = a.part + ((size_t)grp * a.S * 8 + w) * FRAG + lane * 4;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) *(floatx4*)(P + (size_t)split * 8 * FRAG + (nt * 4 + mt) * 256) = acc[nt][mt];
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
      if (!a.xcd) __threadfence();  // splits on different XCDs: write back through L2
      const unsigned prev = atomicAdd(&a.counters[grp], 1u);
      is_last = prev == (unsigned)(a.S - 1);
      if (is_last && !a.xcd) __threadfence();
    }
    __syncthreads();
    if (!is_last) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) acc[nt][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.S; ++sp) {
      floatx4 v[NT][4];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) v[nt][mt] = *(const floatx4*)(P + (size_t)sp * 8 * FRAG + (nt * 4 + mt) * 256);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[nt][mt] += v[nt][mt];
    }
    if (tid == 0) a.counters[grp] = 0u;
  }
  t8_epilogue<NT>(a, ft / (4 * NT), ft, r0, acc, rscale, sq_red, xs + (size_t)(nst % T8_STAGES) * (T8_STAGE_BYTES / 2));
}

// the 128 x 256 LDS-DMA tiles where they apply (SSD_GEMM_T8=0 keeps every
// plan on the 128 x 128 tiles, for comparisons)
static bool tile8_enabled() {
  static const bool on = [] {
    const char* v = std::getenv("SSD_GEMM_T8");
    return !(v && std::strcmp(v, "0") == 0);
  }();
  return on;
}
// the 128 x 192 tiles where they fill a grid better (SSD_GEMM_T8N=0: never)
static bool tile8_narrow_enabled() {
  static const bool on = [] {
    const char* v = std::getenv("SSD_GEMM_T8N");
    return !(v && std::strcmp(v, "0") == 0);
  }();
  return on;
}

GemmPlan gemm_plan_bf16(int M, int N, int K, int xcd) {
  GemmPlan p;
  p.xcd = xcd;
  p.tile = 0;
  p.tail_fb = 0;
  p.tail_S = 1;
  p.tail_nt = 0;
  if (M > 64 && K % (2 * TILE_KT) == 0 && N % 256 == 0 && (size_t)N * K * 2 < (1ull << 31) && tile8_enabled()) {
    // 128 x 256 tiles, eight waves, both operands by LDS DMA, one workgroup
    // per CU: K split by the largest divisor of the stage count that keeps
    // the grid within 256 workgroups, wherever each workgroup still runs at
    // least 32 stages.  Measured on the 8B shapes at 512 rows against the
    // 128 x 128 tiles: gate/up 269 -> 231 us, down 167 -> 122, output layer
    // 274 -> 234, QKV 82 -> 77; O (16 stages per workgroup) 55 -> 62, so it
    // stays on them.
    const int mt = (M + TILE_ROWS - 1) / TILE_ROWS;
    const int nfb = N / 256, nst = K / TILE_KT;
    int S = 1;
    for (int s = 2; s <= 16; ++s)
      if (nst % s == 0 && (long)nfb * mt * s <= 256) S = s;
    if (nst / S >= 32) {
      p.tile = 3;
      p.NT = 4;
      p.MT = TILE_ROWS / 16;
      p.WV = T8_THREADS / 64;
      p.bn = 256;
      p.n_fb = nfb;
      p.m_tiles = mt;
      p.S = S;
      p.KCB = TILE_KT / 32;
      p.kchunks = nst / S;
      p.depth = T8_STAGES;  // ring stages
      // 128 x 192 tiles (waves of 64 x 48) where the 256-feature grid leaves
      // CUs idle and the narrower one fills more of them with no more stages
      // per workgroup (8B QKV: 96 tiles in two splits on 192 CUs at 512 rows,
      // 128 in two splits on all 256 instead).  Only where N > K, which keeps
      // them off the residual projections (N = d, K >= d), whose per-row x^2
      // parts count 256-feature blocks.
      const bool narrow = tile8_narrow_enabled() && N > K;
      if (narrow && N % 192 == 0) {
        const int nfb3 = N / 192;
        int S3 = 0;
        for (int s = 1; s <= 16; ++s)
          if (nst % s == 0 && (long)nfb3 * mt * s <= 256 && nst / s >= 32) S3 = s;
        if (S3 && nst / S3 <= nst / S && (long)nfb3 * mt * S3 > (long)nfb * mt * S) {
          p.NT = 3;
          p.bn = 192;
          p.n_fb = nfb3;
          p.S = S3;
          p.kchunks = nst / S3;
          return p;
        }
      }
      // whole tiles in as many full rounds of 256 as there are, the feature
      // blocks left over K-split so that they fill the last round, where
      // that saves the busiest CU a quarter of a round and more (8B gate/up
      // at 1024 rows: 768 tiles, then 128 in two splits of 32 stages); where
      // no split fits, as 128 x 192 tiles if those fill more of the round
      // (8B gate/up at 512 rows: 256 tiles, then 192 of 256 features as 256
      // of 192)
      const long tiles = (long)nfb * mt, full = tiles / 256;
      if (S == 1 && full >= 1 && tiles % 256 && (256 * full) % mt == 0) {
        const int fb_a = (int)(256 * full / mt), r = (nfb - fb_a) * mt;
        int st = 1;
        for (int s = 2; s <= 16; ++s)
          if (nst % s == 0 && (long)r * s <= 256 && nst / s >= 16) st = s;
        const int fr = (nfb - fb_a) * 256;
        if (st > 1 && nst / st + nst / 8 <= nst * 3 / 4) {
          p.tail_fb = fb_a;
          p.tail_S = st;
        } else if (narrow && fr % 192 == 0 && (long)(fr / 192) * mt <= 256 && (long)(fr / 192) * mt > r) {
          p.tail_fb = fb_a;
          p.tail_nt = 3;
        }
      }
      return p;
    }
  }
  if (M > 64 && K % (2 * TILE_KT) == 0 && N % 64 == 0 && (size_t)N * K * 2 < (1ull << 31)) {
    // 128-feature tiles wherever they give at least 160 workgroups (measured
    // on the 8B and 1B shapes: up to 35 % faster than 64-feature tiles
    // there, slower on grids that leave CUs idle); then K splits until the
    // grid has 256 workgroups
    const int mt = (M + TILE_ROWS - 1) / TILE_ROWS;
    const long w4 = (long)(N / 128) * mt;
    const bool four = N % 128 == 0 && w4 >= 160;
    p.tile = 1;
    p.NT = four ? 4 : 2;
    p.MT = TILE_ROWS / 16;
    p.WV = 4;
    p.bn = 32 * p.NT;
    p.n_fb = N / p.bn;
    p.m_tiles = mt;
    // the split: the smallest divisor of the stage count (at most 16, an
    // even count of stages per split) that brings the grid to 256
    // workgroups, else the largest such divisor (1B down projection at 128
    // rows: 88 stages in 11 splits, 352 workgroups)
    p.S = 1;
    const int nst = K / TILE_KT;
    for (int s = 2; s <= 16 && (long)p.n_fb * mt * p.S < 256; ++s)
      if (nst % s == 0 && (nst / s) % 2 == 0) p.S = s;
    p.KCB = TILE_KT / 32;
    p.kchunks = nst / p.S;
    // four-stage pipeline for 64-feature tiles (measured on the 8B shapes at
    // 512 rows: O 75 -> 59 us, down 241 -> 177); 128-feature tiles would need
    // one workgroup per CU for it, which measured slower
    p.depth = p.NT == 4 ? 3 : (p.kchunks % 4 == 0 ? 4 : 2);
    return p;
  }
  // up to 64 tokens (and shapes the tiled kernel does not take): one-burst
  // launches over row tiles of at most 64 (the weights are streamed once per
  // tile); beyond 128: double-buffered chunks of 128-row tiles
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
  if (p.tile && p.tail_fb) return p.tail_nt ? 0 : (size_t)p.tail_S * (p.n_fb - p.tail_fb) * p.m_tiles * TILE_ROWS * p.bn;
  if (p.S <= 1) return 0;
  if (p.tile) return (size_t)p.S * p.m_tiles * TILE_ROWS * p.n_fb * p.bn;
  (void)M;
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
  if (p.tile) {
    // buffer addressing reaches 2 GiB from each plane's base: rows beyond
    // that go to further launches (chunks of whole row tiles)
    const size_t row_b = (size_t)ld_in * 2;
    int rows = (int)std::min<size_t>((size_t)M, ((1ull << 31) - (size_t)K * 2) / row_b);
    rows = std::max(TILE_ROWS, rows / TILE_ROWS * TILE_ROWS);
    for (int t0 = 0; t0 < M; t0 += rows) {
      GemmKArgs a{};
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
      a.M = std::min(rows, M - t0);
      a.t0 = t0;
      a.xcd = p.xcd;
      a.part = partials;
      a.counters = counters;
      a.epi = epi;
      const dim3 grid(xcd_grid(p.n_fb, (a.M + TILE_ROWS - 1) / TILE_ROWS * p.S, p.xcd));
      if (p.tile == 3 && p.tail_fb && a.M == M) {
        // whole tiles of the first feature blocks, then the rest K-split
        const int mt = (a.M + TILE_ROWS - 1) / TILE_ROWS;
        a.n_fb = p.tail_fb;
        launch_timed(gemm_tile8_kernel<4>, dim3(xcd_grid(a.n_fb, mt, p.xcd)), dim3(T8_THREADS), st, a);
        a.ft0 = p.tail_fb * 16;
        if (p.tail_nt == 3) {
          a.n_fb = (N - p.tail_fb * 256) / 192;
          launch_timed(gemm_tile8_kernel<3>, dim3(xcd_grid(a.n_fb, mt, p.xcd)), dim3(T8_THREADS), st, a);
        } else {
          a.n_fb = p.n_fb - p.tail_fb;
          a.S = p.tail_S;
          a.kchunks = K / TILE_KT / p.tail_S;
          launch_timed(gemm_tile8_kernel<4>, dim3(xcd_grid(a.n_fb, mt * a.S, p.xcd)), dim3(T8_THREADS), st, a);
        }
      } else if (p.tile == 3 && p.NT == 3)
        launch_timed(gemm_tile8_kernel<3>, grid, dim3(T8_THREADS), st, a);
      else if (p.tile == 3)
        launch_timed(gemm_tile8_kernel<4>, grid, dim3(T8_THREADS), st, a);
      else if (p.NT == 4)
        launch_timed(gemm_tile_kernel<4, 3>, grid, dim3(256), st, a);
      else if (p.depth == 4)
        launch_timed(gemm_tile_kernel<2, 4>, grid, dim3(256), st, a);
      else
        launch_timed(gemm_tile_kernel<2, 2>, grid, dim3(256), st, a);
    }
    return;
  }
  const int MP = p.MT * 16;
  for (int t0 = 0; t0 < M; t0 += MP) {
    GemmKArgs a;
    a.ft0 = 0;
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
