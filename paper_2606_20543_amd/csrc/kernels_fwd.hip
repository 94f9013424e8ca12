// Persistent forward pass for small token counts (M <= 32 block tokens).
//
// One cooperative launch runs every layer of the backbone (QKV projection with
// rotary embedding and KV write, attention, O projection + residual, gate/up +
// SwiGLU, down projection + residual) and the output layer.  Every phase is a
// list of work items spread over all workgroups (all resident at once), and a
// workgroup moves on as soon as its own items are done: item dependencies are
// tracked with per-unit flags instead of kernel boundaries, so the weights of a
// workgroup's next projection item stream from HBM while the current phase's
// reduction tail and the following phase's inputs are still being produced.
//
// Coherence across the 8 XCDs: a producer writes its outputs with agent-scope
// stores (sc1, written through the XCD's L2), waits for them, then stores the
// unit's flag (agent scope); a consumer polls the flags it needs with
// agent-scope loads and then reads the data with agent-scope loads.  Split-K
// partials and attention chunk partials stay inside one XCD's L2 (the members
// of a reduction group run on one XCD).  Flags carry the value
// epoch * (layers + 1) + layer + 1, so they never need resetting.  Every wait is
// bounded: a wait that runs out sets an abort flag, after which every later wait
// gives up at once, so the grid always drains; the host reports the abort.
#include "tiles.h"

namespace ssd {

namespace {

constexpr int FWD_THREADS = 256;
constexpr int FWD_KCB = 16;  // k-blocks of 32 per GEMM item (one burst)
constexpr int FWD_RMS_PARTS = 64;  // rms partial sums per token (d_model <= 4096)

__device__ __forceinline__ unsigned ld_flag(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wave-cooperative wait (call from all 64 lanes of one wave): flags[u] >= val
// for every u in [lo, hi).  Returns false when the wait was abandoned.
__device__ bool wait_units(const unsigned* flags, int lo, int hi, unsigned val, unsigned* abort_flag,
                           unsigned spin_limit) {
  const int lane = threadIdx.x & 63;
  for (int base = lo; base < hi; base += 64) {
    const int u = base + lane;
    const unsigned* fp = flags + (u < hi ? u : lo);
    unsigned n = 0;
    while (true) {
      const bool ok = u >= hi || ld_flag(fp) >= val;
      if (__builtin_amdgcn_uicmp((int)!ok, 0, 33) == 0) break;  // no lane still waiting
      ++n;
      if (n > spin_limit || ((n & 255) == 0 && ld_flag(abort_flag))) {
        if (lane == 0) __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return false;
      }
      __builtin_amdgcn_s_sleep(2);
    }
  }
  return true;
}

}  // namespace

// Workgroup-level wait on up to three flag ranges; all threads call it.
// Returns false (for every thread) if the pass is being abandoned.
__device__ bool wg_wait(const unsigned* f0, int lo0, int hi0, const unsigned* f1, int lo1, int hi1,
                        const unsigned* f2, int lo2, int hi2, unsigned val, const FwdArgs& A, int* sflag) {
  if (threadIdx.x < 64) {
    bool ok = ld_flag(A.abort_flag) == 0u;
    if (ok && f0) ok = wait_units(f0, lo0, hi0, val, A.abort_flag, A.spin_limit);
    if (ok && f1) ok = wait_units(f1, lo1, hi1, val, A.abort_flag, A.spin_limit);
    if (ok && f2) ok = wait_units(f2, lo2, hi2, val, A.abort_flag, A.spin_limit);
    if (threadIdx.x == 0) *sflag = ok ? 1 : 0;
  }
  lds_barrier();
  const bool ok = *sflag != 0;
  lds_barrier();  // every thread has read the flag before it is reused
  return ok;
}

// LDS of one workgroup: the union of the GEMM and attention stages.
template <int MT, int D>
struct FwdLds {
  using X = XStage<MT, FWD_KCB>;
  static constexpr int GEMM_BYTES = 2 * X::PL * 2 + (4 * X::MP + X::MP + 256) * 4;
  static constexpr int ATT_ROWS = 16;  // one query tile per workgroup
  static constexpr int ATT_Q_OFF = (AtShape<1>::WAVES * ATT_ROWS * (D + 4) + 2 * AtShape<1>::WAVES * ATT_ROWS) * 4;
  static constexpr int ATT_BYTES = ATT_Q_OFF + (D / 32) * 2 * 1024;  // + the query tiles
  static_assert(ATT_Q_OFF % 16 == 0, "query stage 16-byte aligned");
  static constexpr int BYTES = GEMM_BYTES > ATT_BYTES ? GEMM_BYTES : ATT_BYTES;
};

// The phase table is read through the constant address space: the kernel
// never writes it, so its fields come in through scalar loads (lgkmcnt).  A
// generic pointer would make them vector loads, and every wait for one of
// those would also wait for the workgroup's weight stream in flight.
#if defined(__HIP_DEVICE_COMPILE__)
typedef const __attribute__((address_space(4))) FwdPhase* PhaseTab;
#else
typedef const FwdPhase* PhaseTab;  // host pass: device code is parsed, not generated
#endif
__device__ __forceinline__ PhaseTab phase_tab(const FwdArgs& A) { return (PhaseTab)(uintptr_t)A.phases; }

// this workgroup's first item of a phase rotated by rot
__device__ __forceinline__ int first_item(int rot) {
  const int G = gridDim.x;
  return ((int)blockIdx.x - rot + G) % G;
}

// Next GEMM item of this workgroup after item `it` of phase p (it < 0: none
// in p), not looking past an attention phase (the prefetched weights are not
// kept live across the attention code): (p2, it2), or p2 = -1.
__device__ __forceinline__ void next_gemm_item(const FwdArgs& A, int p, int it, int& p2, int& it2) {
  const int G = gridDim.x;
  const PhaseTab tab = phase_tab(A);
  if (p >= 0 && it >= 0 && tab[p].kind == FWD_GEMM && it + G < tab[p].g.items) {
    p2 = p;
    it2 = it + G;
    return;
  }
  for (int q = p + 1; q < A.n_phases; ++q) {
    if (tab[q].kind != FWD_GEMM) break;
    const int first = first_item(tab[q].rot);
    if (first < tab[q].g.items) {
      p2 = q;
      it2 = first;
      return;
    }
  }
  p2 = -1;
}

// weights of burst b (16 k-blocks) of item `it` of phase p
template <int MT>
__device__ __forceinline__ void issue_weights(PhaseTab tab, int p, int it, int b, int xcd, u32x4 (&ra)[1][FWD_KCB]) {
  const int S = tab[p].g.S, n_fb = tab[p].g.n_fb;
  int fb, s;
  xcd_unmap(it, S, xcd, fb, s);
  if (fb >= n_fb) fb = n_fb - 1;  // idle slot: any valid tile (never used)
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  load_a<1, FWD_KCB>(ra, (const u32x4*)tab[p].g.W, tab[p].g.KB, fb * 4 + w, tab[p].g.N,
                     (s * tab[p].g.bursts + b) * FWD_KCB, lane);
}

// One GEMM work item (feature block fb, K-split s of g.bursts 512-wide
// bursts).  The first burst's weights are in ra (loaded by the caller); the
// later ones are loaded here, each after the previous burst's products.
// Returns whether this workgroup ran the epilogue.
template <int MT>
__device__ __forceinline__ void gemm_item(const FwdArgs& A, PhaseTab tab, int p, const FwdGemm& g, int it,
                                          u32x4 (&ra)[1][FWD_KCB], unsigned char* smem, int* sflag, bool& last) {
  using X = XStage<MT, FWD_KCB>;
  uint16_t* xs = (uint16_t*)smem;
  float* sq_red = (float*)(smem + 2 * X::PL * 2);  // [4][MP]
  float* rscale = sq_red + 4 * X::MP;              // [MP]
  float* rms_red = rscale + X::MP;                 // [256]
  int fb, s;
  xcd_unmap(it, g.S, A.xcd, fb, s);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nb0 = fb * 4 + w;
  const EpiArgs& e = g.epi;
  const unsigned val = A.epoch_base + (unsigned)g.dep_layer;

  // inputs of this K-slice: the producer units covering [s*KC, (s+1)*KC) (x dep_scale)
  const int KC = FWD_KCB * 32 * g.bursts;
  int u0 = 0, u1 = g.dep_units;
  if (g.dep_att) {
    // attention outputs: the query groups of the KV heads whose query heads
    // this slice covers (one sequence; several sequences wait for all groups)
    const AttnKArgs& at = A.att;
    if (at.heads == at.Hkv) {
      const int h0 = (s * KC) / e.D, h1 = ((s + 1) * KC - 1) / e.D;
      u0 = (h0 / at.g) * at.nqg;
      u1 = (h1 / at.g + 1) * at.nqg;
    } else {
      u1 = at.groups;
    }
  } else if (g.dep_units == 0) {
    u0 = (s * KC * g.dep_scale) / g.dep_width;
    u1 = ((s + 1) * KC * g.dep_scale + g.dep_width - 1) / g.dep_width;
  }
  EpiOps<1, MT> op;
  epi_block_starts<1, MT>(e, g.M, 0, lane, op);
  if (!wg_wait(g.dep, u0, u1, nullptr, 0, 0, nullptr, 0, 0, val, A, sflag)) {
    last = false;
    return;
  }
  floatx4 acc[1][MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[0][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int b = 0; b < g.bursts; ++b) {
    if (b > 0) {
      lds_barrier();  // every wave is done reading the previous x chunk
      issue_weights<MT>(tab, p, it, b, A.xcd, ra);
    }
    load_x_lds<MT, FWD_KCB, CPOL_SC1>(xs, g.in, g.in_plane, g.ld_in, g.M, s * KC + b * FWD_KCB * 32);
    __builtin_amdgcn_s_waitcnt(0);  // this wave's LDS copies (and its weight loads) have landed
    lds_barrier();
    compute_chunk<MT, 1, FWD_KCB>(acc, ra, xs, lane);
  }

  const size_t frag = (size_t)MT * 64 * 4;
  const size_t P = ((size_t)fb * 4 + w) * frag;  // this wave's fragment (floats from g.part)
  const size_t split_stride = (size_t)g.n_fb * 4 * frag;
  if (g.S > 1) {
    // partials stay in this XCD's L2; the reading side skips L1, which may
    // still hold the lines from an earlier layer's reduction
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const floatx4 v = acc[0][mt];
      XcdMem::stf4(g.part, (P + (size_t)s * split_stride + (mt * 64 + lane) * 4) * 4,
                   make_float4(v[0], v[1], v[2], v[3]));
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
      if (!A.xcd) __threadfence();
      const unsigned prev = atomicAdd(&g.counters[fb], 1u);
      const bool lst = prev == (unsigned)(g.S - 1);
      if (lst) {
        // every split has arrived: re-arm the counter for the next pass
        __hip_atomic_store(&g.counters[fb], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (!A.xcd) __threadfence();
      }
      *sflag = lst;
    }
    __syncthreads();
    last = *sflag != 0;
    __syncthreads();
    if (!last) return;
  } else {
    last = true;
  }
  // epilogue: the rms partial sums must be complete
  if (g.rms_dep && !wg_wait(g.rms_dep, 0, g.rms_units, nullptr, 0, 0, nullptr, 0, 0, A.epoch_base + (unsigned)g.rms_layer, A,
                            sflag))
    return;
  epi_load<1, MT, CoherentMem>(e, nb0, g.N, g.M, 0, lane, op);
  float rv[RmsPre<X::MP, FWD_RMS_PARTS>::RQ];
  rms_issue<X::MP, CoherentMem, FWD_RMS_PARTS>(e, g.in, g.M, 0, rv);
  if (g.S > 1) {
    const size_t Pl = P + lane * 4;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[0][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < g.S; s0 += 4) {
      floatx4 pv[4][MT];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const size_t Ps = Pl + (size_t)min(s0 + j, g.S - 1) * split_stride;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const float4 v = XcdMem::ldf4(g.part, (Ps + mt * 64 * 4) * 4);
          pv[j][mt] = floatx4{v.x, v.y, v.z, v.w};
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float m = (s0 + j < g.S) ? 1.f : 0.f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[0][mt] += pv[j][mt] * m;
      }
    }
  }
  rms_finish<X::MP, FWD_RMS_PARTS>(e, rv, rms_red, rscale);
  lds_barrier();
  float sq[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) sq[mt] = 0.f;
  epi_store<1, MT, CoherentMem>(e, acc, op, nb0, g.N, g.M, 0, lane, rscale, sq);
  if (e.kind == EPI_RESID) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) sq_red[w * X::MP + mt * 16 + lane] = v;
    }
    __syncthreads();
    if (threadIdx.x < X::MP && threadIdx.x < g.M) {
      const int tl = threadIdx.x;
      const float v = ((sq_red[tl] + sq_red[X::MP + tl]) + sq_red[2 * X::MP + tl]) + sq_red[3 * X::MP + tl];
      __hip_atomic_store(&e.ssq_out[(size_t)fb * e.ssq_out_ld + tl], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  // outputs complete at agent scope, then the unit's flag
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (g.out_flags)
      __hip_atomic_store(&g.out_flags[fb], A.epoch_base + (unsigned)g.out_layer, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <int MT, int D>
__global__ __launch_bounds__(FWD_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2))) void fwd_kernel(FwdArgs A) {
  __shared__ __align__(16) unsigned char smem[FwdLds<MT, D>::BYTES];
  __shared__ int sflag;
  const PhaseTab tab = phase_tab(A);
  if (A.probe && threadIdx.x == 0)
    A.probe[blockIdx.x] = (int)(__builtin_amdgcn_s_getreg(20 | (0 << 6) | ((4 - 1) << 11)) & 0xF);  // XCC_ID
  u32x4 ra[1][FWD_KCB];
  int pre_p = -1, pre_it = -1;  // the item whose weights ra holds (or is loading)
  {
    int p2, it2;
    next_gemm_item(A, -1, 0, p2, it2);
    if (p2 >= 0) {
      issue_weights<MT>(tab, p2, it2, 0, A.xcd, ra);
      pre_p = p2;
      pre_it = it2;
    }
  }
  for (int p = 0; p < A.n_phases; ++p) {
    const FwdPhase ph = tab[p];  // by value: the fields live in scalar registers
    if (ph.kind == FWD_GEMM) {
      const FwdGemm& g = ph.g;
      for (int it = first_item(ph.rot); it < g.items; it += gridDim.x) {
        int fb, s;
        xcd_unmap(it, g.S, A.xcd, fb, s);
        if (!(pre_p == p && pre_it == it)) issue_weights<MT>(tab, p, it, 0, A.xcd, ra);
        pre_p = -1;
        bool last = false;
        if (fb < g.n_fb) gemm_item<MT>(A, tab, p, g, it, ra, smem, &sflag, last);
        // next item's weights: right away for a workgroup that ran no
        // epilogue, after the epilogue otherwise (its loads must not queue
        // behind a weight burst)
        int p2, it2;
        next_gemm_item(A, p, it, p2, it2);
        if (p2 >= 0) {
          issue_weights<MT>(tab, p2, it2, 0, A.xcd, ra);
          pre_p = p2;
          pre_it = it2;
        }
        (void)last;
      }
    } else {
      const FwdAttn& at = ph.a;
      float* sm_o = (float*)smem;
      float* sm_m = sm_o + AtShape<1>::WAVES * 16 * (D + 4);
      float* sm_l = sm_m + AtShape<1>::WAVES * 16;
      for (int it = first_item(ph.rot); it < A.att_items; it += gridDim.x) {
        // inputs: q of the group's query heads, k and v of its KV head
        int z, qg, grp_id, c;
        if (A.att.nchunk == 1) {
          xcd_unmap(it, A.att.nqg, A.att.xcd, z, qg);
        } else {
          xcd_unmap(it, A.att.nchunk, A.att.xcd, grp_id, c);
          z = grp_id / A.att.nqg;
        }
        if (z >= A.att.heads) continue;
        const int hkv = z % A.att.Hkv;
        const int uq0 = hkv * A.att.g * D / at.dep_width, uq1 = (hkv + 1) * A.att.g * D / at.dep_width;
        const int uk0 = (at.qN + hkv * D) / at.dep_width, uk1 = (at.qN + (hkv + 1) * D) / at.dep_width;
        const int uv0 = (at.qN + at.kN + hkv * D) / at.dep_width, uv1 = (at.qN + at.kN + (hkv + 1) * D) / at.dep_width;
        if (!wg_wait(at.dep, uq0, uq1, at.dep, uk0, uk1, at.dep, uv0, uv1, A.epoch_base + (unsigned)at.layer, A, &sflag))
          continue;
        AttnKArgs a = A.att;
        a.kc = (const uint16_t*)at.kc;
        a.vc = (const uint16_t*)at.vc;
        const int done = attn_unit<D, 1, CoherentMem, false, XcdMem, true>(
            a, it, sm_o, sm_m, sm_l, &sflag, (uint16_t*)(smem + FwdLds<MT, D>::ATT_Q_OFF));
        if (done >= 0) {
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          if (threadIdx.x == 0)
            __hip_atomic_store(&at.out_flags[done], A.epoch_base + (unsigned)at.layer, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();
      }
      // the following projection's weights, now that the attention is done
      // (ra is redefined on every path, so it is dead across the attention)
      int p2, it2;
      next_gemm_item(A, p, -1, p2, it2);
      if (p2 >= 0) {
        issue_weights<MT>(tab, p2, it2, 0, A.xcd, ra);
        pre_p = p2;
        pre_it = it2;
      } else {
#pragma unroll
        for (int i = 0; i < FWD_KCB; ++i) ra[0][i] = u32x4{0u, 0u, 0u, 0u};
        pre_p = -1;
      }
    }
  }
  // a prefetch past the last phase cannot exist (next_gemm_item finds none);
  // drain anything still in flight before the registers die
  __builtin_amdgcn_s_waitcnt(0);
}

template <int MT, int D>
static hipError_t launch_fwd(const FwdArgs& a, int grid, hipStream_t st) {
  void* args[] = {(void*)&a};
  // a cooperative launch takes no dispatch events: a timed launch is bracketed
  // by event records (negligible next to a whole forward pass)
  hipEvent_t t0 = nullptr, t1 = nullptr;
  if (g_launch_timer) {
    g_launch_timer->next(t0, t1);
    hipError_t e = hipEventRecord(t0, st);
    if (e != hipSuccess) return e;
  }
  hipError_t e = hipLaunchCooperativeKernel((const void*)fwd_kernel<MT, D>, dim3(grid), dim3(FWD_THREADS), args, 0, st);
  if (e == hipSuccess && t1) e = hipEventRecord(t1, st);
  return e;
}

hipError_t fwd_persistent(const FwdArgs& a, int MT, int D, int grid, hipStream_t st) {
  if (MT == 1) return D == 128 ? launch_fwd<1, 128>(a, grid, st) : launch_fwd<1, 64>(a, grid, st);
  return D == 128 ? launch_fwd<2, 128>(a, grid, st) : launch_fwd<2, 64>(a, grid, st);
}

int fwd_max_grid(int MT, int D) {
  int per_cu = 0, ncu = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  int coop = 0;
  if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess || !coop) return 0;
  const void* k = MT == 1 ? (D == 128 ? (const void*)fwd_kernel<1, 128> : (const void*)fwd_kernel<1, 64>)
                          : (D == 128 ? (const void*)fwd_kernel<2, 128> : (const void*)fwd_kernel<2, 64>);
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, FWD_THREADS, 0) != hipSuccess) return 0;
  return per_cu * ncu;
}

}  // namespace ssd
