// Device building blocks shared by the GEMM, attention and persistent
// forward kernels (gfx950): MFMA operand tiles, token staging through LDS,
// fused GEMM epilogues and the per-block attention step.  Memory accesses to
// activations go through a policy: PlainMem (ordinary loads and stores, for
// kernels whose producers finished in an earlier launch) or CoherentMem
// (agent-scope accesses, sc1, which bypass the per-XCD L2 so that producers
// and consumers on different XCDs of one running kernel see each other's
// data without L2 write-back or invalidation).
#pragma once

#include <type_traits>
#include <utility>

#include "ssd_internal.h"

namespace ssd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// Two fp32 values -> a packed bf16 pair (a in the low half) by gfx950's
// packed conversion: round to nearest even, the same bits as f2bf on each
// finite value, in one instruction instead of about six.
__device__ __forceinline__ uint32_t cvt2bf(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// ---- LDS DMA pipelines ----
// s_waitcnt with only vmcnt (six bits on gfx9) counted; expcnt and lgkmcnt left alone
template <int V>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(V >= 0 && V < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((V & 15) | (7 << 4) | (15 << 8) | ((V >> 4) << 14));
}

// Workgroup barrier of an LDS DMA pipeline.  A release fence would make the
// compiler drain every LDS DMA copy in flight (vmcnt(0)), also those of the
// steps copied ahead; each wave waits for its own copies of the step about to
// be read (wait_vmcnt) and the barrier orders the rest.  The memory clobber
// keeps LDS accesses on their side of it.
__device__ __forceinline__ void dma_barrier() { asm volatile("s_barrier" ::: "memory"); }

// 16 bytes per lane from buffer r at (voff + soff) into LDS at lds + 16 * lane
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint16_t* lds, int voff, int soff) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, soff, 0, 0);
#else
  (void)r, (void)lds, (void)voff, (void)soff;
#endif
}

// raw buffer resource over 2 GiB from b
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* b) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(b), 0, 0x7FFFFFFF, 0x00020000);
}

// LDS byte address of a pointer into a __shared__ array
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// 16-byte LDS read at a constant byte offset from addr (the instruction's
// offset field), issued as an instruction of its own.  The compiler would
// make a plain LDS load wait for every LDS DMA copy in flight (it cannot tell
// which LDS bytes a copy writes), which drains the copies of the blocks
// fetched ahead; these reads are ordered by lgkm_wait instead, and the
// barrier of each step keeps them clear of the copies into the same buffer.
template <int OFF>
__device__ __forceinline__ u32x4 ds_read16_at(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds_read offset field");
  u32x4 v;
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
#else
  (void)addr;
  v = u32x4{0u, 0u, 0u, 0u};
#endif
  return v;
}

// 1 KiB tiles FIRST .. FIRST + N - 1 of the LDS block at addr into dst[0 .. N - 1]
template <int FIRST, int... I>
__device__ __forceinline__ void ds_read_tiles(u32x4* dst, uint32_t addr, std::integer_sequence<int, I...>) {
  ((dst[I] = ds_read16_at<(FIRST + I) * 1024>(addr)), ...);
}

// waits until at most min(n, MAXB) groups of PER loads of this wave are
// outstanding (n known only at run time; vmcnt takes an immediate)
template <int PER, int MAXB>
__device__ __forceinline__ void wait_vm_groups(int n) {
  if constexpr (MAXB == 0) {
    (void)n;
    wait_vmcnt<0>();
  } else {
    if (n >= MAXB)
      wait_vmcnt<MAXB * PER>();
    else
      wait_vm_groups<PER, MAXB - 1>(n);
  }
}

// waits until at most N LDS operations of this wave are outstanding; the
// registers passed are tied to the wait, so no use of them moves above it
template <int N, int R>
__device__ __forceinline__ void lgkm_wait(u32x4 (&r)[R]) {
#if defined(__HIP_DEVICE_COMPILE__)
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  if constexpr (R == 3)
    asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]) : "n"(N));
  else if constexpr (R == 4)
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]) : "n"(N));
  else if constexpr (R == 8)
    asm volatile("s_waitcnt lgkmcnt(%8)"
                 : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]), "+v"(r[7])
                 : "n"(N));
  else
    static_assert(R == 3 || R == 4 || R == 8, "register groups of 3, 4 or 8");
#else
  (void)r;
#endif
}

// Every access names a base pointer and a byte offset from it.  The base is
// wave-uniform at every call site (a kernel argument or a field of one), which
// lets CoherentMem address through a buffer resource built from it.
struct PlainMem {
  template <typename T>
  static __device__ __forceinline__ const T* at(const void* b, size_t off) {
    return (const T*)((const char*)b + off);
  }
  template <typename T>
  static __device__ __forceinline__ T* at(void* b, size_t off) {
    return (T*)((char*)b + off);
  }
  static __device__ __forceinline__ u32x4 ld16(const void* b, size_t off) { return *at<u32x4>(b, off); }
  static __device__ __forceinline__ float ld4f(const void* b, size_t off) { return *at<float>(b, off); }
  static __device__ __forceinline__ float4 ldf4(const void* b, size_t off) { return *at<float4>(b, off); }
  static __device__ __forceinline__ float2 ldf2(const void* b, size_t off) { return *at<float2>(b, off); }
  static __device__ __forceinline__ void st2(void* b, size_t off, uint16_t v) { *at<uint16_t>(b, off) = v; }
  static __device__ __forceinline__ void st4(void* b, size_t off, uint32_t v) { *at<uint32_t>(b, off) = v; }
  static __device__ __forceinline__ void st8(void* b, size_t off, uint2 v) { *at<uint2>(b, off) = v; }
  static __device__ __forceinline__ void stf4(void* b, size_t off, float4 v) { *at<float4>(b, off) = v; }
  static __device__ __forceinline__ void stf2(void* b, size_t off, float2 v) { *at<float2>(b, off) = v; }
  static constexpr int LDS_AUX = 0;  // cache policy of LDS DMA reads
};

// Buffer-instruction accesses with a cache policy (raw buffer, 2 GiB range
// from the base; callers keep offsets below that).  Unlike atomic loads these
// are ordinary memory operations: the compiler issues them back to back.
template <int LD_POL, int ST_POL>
struct BufMem {
  static constexpr int LDS_AUX = LD_POL;
  // the base is uniform by contract; readfirstlane keeps it in scalar
  // registers where the compiler cannot prove that (no per-lane loop)
  static __device__ __forceinline__ __amdgpu_buffer_rsrc_t rs(const void* b) {
    const uint64_t a = (uint64_t)b;
    const uint64_t u = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
                       (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
    return __builtin_amdgcn_make_buffer_rsrc((void*)u, 0, 0x7FFFFFFF, 0x00020000);
  }
  static __device__ __forceinline__ u32x4 ld16(const void* b, size_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(rs(b), (int)off, 0, LD_POL);
  }
  static __device__ __forceinline__ float ld4f(const void* b, size_t off) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs(b), (int)off, 0, LD_POL));
  }
  static __device__ __forceinline__ float4 ldf4(const void* b, size_t off) {
    const u32x4 v = ld16(b, off);
    return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w));
  }
  static __device__ __forceinline__ float2 ldf2(const void* b, size_t off) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rs(b), (int)off, 0, LD_POL);
    return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
  }
  static __device__ __forceinline__ void st2(void* b, size_t off, uint16_t v) {
    __builtin_amdgcn_raw_buffer_store_b16(v, rs(b), (int)off, 0, ST_POL);
  }
  static __device__ __forceinline__ void st4(void* b, size_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b32(v, rs(b), (int)off, 0, ST_POL);
  }
  static __device__ __forceinline__ void st8(void* b, size_t off, uint2 v) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{v.x, v.y}, rs(b), (int)off, 0, ST_POL);
  }
  static __device__ __forceinline__ void stf4(void* b, size_t off, float4 v) {
    __builtin_amdgcn_raw_buffer_store_b128(
        u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)}, rs(b),
        (int)off, 0, ST_POL);
  }
  static __device__ __forceinline__ void stf2(void* b, size_t off, float2 v) {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(v.x), __float_as_uint(v.y)}, rs(b), (int)off, 0,
                                          ST_POL);
  }
};
// cache-policy bits of gfx950 vector memory instructions
constexpr int CPOL_SC0 = 1;   // loads: miss in the CU's L1 (read from the XCD's L2)
constexpr int CPOL_SC1 = 16;  // device scope: coherent across the XCDs' L2s (write-through stores)
// Data exchanged between workgroups on any XCDs inside one running kernel.
using CoherentMem = BufMem<CPOL_SC1, CPOL_SC1>;
// Data exchanged inside one XCD (split-K and key-chunk partials): plain stores
// land in the XCD's L2, loads skip the CU's L1 (which may still hold the lines
// from an earlier use of the same buffer in the same kernel).
using XcdMem = BufMem<CPOL_SC0, 0>;

template <int NT, int KCB>
__device__ __forceinline__ void load_a(u32x4 (&ra)[NT][KCB], const u32x4* W, int KB, int nb0, int N, int kb0,
                                       int lane) {
  // feature tiles past N reload the last tile (no branch: a branch around the
  // burst makes the compiler wait for all of it at the join); their results
  // are never stored
  const u32x4* p[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int nb = (nb0 + nt) * 16 < N ? nb0 + nt : N / 16 - 1;
    p[nt] = W + ((size_t)nb * KB + kb0) * 64 + lane;
  }
  // issued in the order the MFMAs consume them (k-block major), each waited
  // for by its position in the queue: no scheduling across the loads
#pragma unroll
  for (int kb = 0; kb < KCB; ++kb)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      ra[nt][kb] = __builtin_nontemporal_load(p[nt] + kb * 64);
      __builtin_amdgcn_sched_barrier(0);
    }
}

template <int MT, int KCB, int NTH = 256>
struct XStage {
  static constexpr int MP = MT * 16;
  static constexpr int KC = KCB * 32;
  static constexpr int LD = KC + 8;          // bf16 per LDS row (16-byte pad)
  static constexpr int PL = MP * LD;         // one plane
  static constexpr int CG = KC / 8;          // 16-byte column groups per row
  static constexpr int RSTEP = NTH / CG;     // rows covered per pass (NTH threads)
  static constexpr int PASSES = (MP + RSTEP - 1) / RSTEP;
};

// x chunk (both planes) -> registers
template <int MT, int KCB, int NP, class Mem = PlainMem, int NTH = 256>
__device__ __forceinline__ void load_x(u32x4 (&rx)[2][NP], const uint16_t* in, size_t plane, int ld_in, int M,
                                       int k0) {
  using X = XStage<MT, KCB, NTH>;
  const int cg = threadIdx.x % X::CG, r0 = threadIdx.x / X::CG;
  // token rows past M repeat row M-1: no branch around the loads (so they
  // issue back to back); the results of those rows are never stored
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const int r = r0 + p * X::RSTEP;
    const int rc = r < M ? r : M - 1;
    const size_t off = ((size_t)rc * ld_in + k0 + cg * 8) * 2;
    rx[0][p] = Mem::ld16(in, off);
    rx[1][p] = Mem::ld16(in, off + plane * 2);
  }
}

// The same chunk straight into LDS (gfx950 LDS DMA, 16 bytes per lane, no
// registers): wave w copies rows w, w + 4, ... of both planes, one 1 KiB row
// per instruction.  AUX: cache policy of the global reads.  The caller waits
// for vmcnt(0) and then barriers before the LDS is read.
template <int MT, int KCB, int AUX, int NW = 4>
__device__ __forceinline__ void load_x_lds(uint16_t* xs, const uint16_t* in, size_t plane, int ld_in, int M, int k0) {
  using X = XStage<MT, KCB>;
  static_assert(X::KC == 512, "one 512-input row per wave instruction");
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
  for (int r = w; r < X::MP; r += NW) {
    if (r >= M) break;  // rows past M are never stored (their LDS rows stay stale)
    const uint16_t* src = in + (size_t)r * ld_in + k0 + lane * 8;
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                     (void __attribute__((address_space(3)))*)(xs + r * X::LD), 16, 0, AUX);
    __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)(src + plane),
                                     (void __attribute__((address_space(3)))*)(xs + X::PL + r * X::LD), 16, 0, AUX);
  }
}

template <int MT, int KCB, int NP, int NTH = 256>
__device__ __forceinline__ void store_x(const u32x4 (&rx)[2][NP], uint16_t* xs) {
  using X = XStage<MT, KCB, NTH>;
  const int cg = threadIdx.x % X::CG, r0 = threadIdx.x / X::CG;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    int r = r0 + p * X::RSTEP;
    if (X::PASSES * X::RSTEP == X::MP || r < X::MP) {
      *(u32x4*)(xs + r * X::LD + cg * 8) = rx[0][p];
      *(u32x4*)(xs + X::PL + r * X::LD + cg * 8) = rx[1][p];
    }
  }
}

// k-block order, so the MFMAs of block kb wait only for that block's weights
template <int MT, int NT, int KCB>
__device__ __forceinline__ void compute_chunk(floatx4 (&acc)[NT][MT], const u32x4 (&ra)[NT][KCB], const uint16_t* xs,
                                              int lane) {
  using X = XStage<MT, KCB>;
  const int row = lane & 15, col = (lane >> 4) * 8;
#pragma unroll
  for (int kb = 0; kb < KCB; ++kb) {
    bf16x8 bhi[MT], blo[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const uint16_t* p = xs + (mt * 16 + row) * X::LD + kb * 32 + col;
      bhi[mt] = __builtin_bit_cast(bf16x8, *(const u32x4*)p);
      blo[mt] = __builtin_bit_cast(bf16x8, *(const u32x4*)(p + X::PL));
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      bf16x8 a = __builtin_bit_cast(bf16x8, ra[nt][kb]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bhi[mt], acc[nt][mt], 0, 0, 0);
        acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, blo[mt], acc[nt][mt], 0, 0, 0);
      }
    }
  }
}

// ---- per-token 1/rms(x) from the producer's partial sums of x^2 ----
// Thread (t = tid % MP, part group pg = tid / MP) loads parts pg, pg + G, ...
// into registers before the weight burst is issued (so the wait for them does
// not wait for the weights), sums them in part order, and the G group sums
// meet in LDS (summed in group order: deterministic).
template <int MP, int PARTS = GEMM_RMS_MAX_PARTS, int NTH = 256>
struct RmsPre {
  static constexpr int G = NTH / MP;
  static constexpr int RQ = (PARTS + G - 1) / G;
};

// raw loads only (no use of the values, so nothing waits for them here);
// without partial sums (ssq == nullptr) the loads read in[0] and are ignored
template <int MP, class Mem = PlainMem, int PARTS = GEMM_RMS_MAX_PARTS, int NTH = 256>
__device__ __forceinline__ void rms_issue(const EpiArgs& e, const void* dummy, int M, int t0,
                                          float (&v)[RmsPre<MP, PARTS, NTH>::RQ]) {
  const int t = threadIdx.x % MP, pg = threadIdx.x / MP;
  const int tc = t < M ? t : M - 1;
  const bool has = e.ssq != nullptr;
  const float* base = has ? e.ssq : (const float*)dummy;
  const size_t c = has ? (size_t)e.ssq_off + (size_t)(t0 + tc) * e.ssq_step : 0;
  const size_t ld = has ? (size_t)e.ssq_ld : 0;
#pragma unroll
  for (int q = 0; q < RmsPre<MP, PARTS, NTH>::RQ; ++q) {
    const int p = pg + q * RmsPre<MP, PARTS, NTH>::G;
    v[q] = Mem::ld4f(base, ((size_t)(p < e.ssq_parts ? p : 0) * ld + c) * 4);
  }
}

// writes rscale[0..MP); visible after the caller's next barrier
template <int MP, int PARTS = GEMM_RMS_MAX_PARTS, int NTH = 256>
__device__ __forceinline__ void rms_finish(const EpiArgs& e, const float (&v)[RmsPre<MP, PARTS, NTH>::RQ], float* red,
                                           float* rscale) {
  // branch-free in ssq (a branch here would make the compiler settle the
  // weight loads at the join); without partial sums the scale is 1
  const int pg = threadIdx.x / MP;
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < RmsPre<MP, PARTS, NTH>::RQ; ++q) s += (pg + q * RmsPre<MP, PARTS, NTH>::G < e.ssq_parts) ? v[q] : 0.f;
  red[threadIdx.x] = s;  // [pg][t]
  lds_barrier();
  if (threadIdx.x < MP) {
    float a = 0.f;
#pragma unroll
    for (int g = 0; g < RmsPre<MP, PARTS, NTH>::G; ++g) a += red[g * MP + threadIdx.x];
    rscale[threadIdx.x] = e.ssq ? 1.0f / sqrtf(a * e.inv_d + e.eps) : 1.f;
  }
}

// sum of parts p0 .. p0 + Q - 1 (those below the part count) of one row, in
// part order, NB loads in flight at a time
template <int NB>
__device__ __forceinline__ float rms_part_sum(const EpiArgs& e, size_t c, int p0, int Q) {
  float s = 0.f;
  for (int b0 = 0; b0 < Q; b0 += NB) {
    float v[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int p = p0 + b0 + j;
      v[j] = e.ssq[(size_t)(p < e.ssq_parts ? p : 0) * e.ssq_ld + c];
    }
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (b0 + j < Q && p0 + b0 + j < e.ssq_parts) s += v[j];
  }
  return s;
}

// per-token 1/rms(x) for large token tiles: the NTH / MP thread groups each
// take a contiguous range of the parts of every row, issue their loads
// together (in batches of 16 where a range is longer: 64 parts over four
// groups are one batch), sum them in part order, and the group sums meet in
// LDS, summed in group order (deterministic).  red: NTH floats of LDS.
template <int MP, int NTH = 256>
__device__ __forceinline__ void rms_prologue(const EpiArgs& e, int M, int t0, float (*red)[MP], float* rscale) {
  constexpr int G = NTH / MP;
  static_assert(G >= 1 && G * MP == NTH, "whole row groups");
  const int t = threadIdx.x % MP, g = threadIdx.x / MP;
  const int tc = t < M ? t : M - 1;
  const int Q = (e.ssq_parts + G - 1) / G;
  const size_t c = (size_t)e.ssq_off + (size_t)(t0 + tc) * e.ssq_step;
  const float s = Q <= 4 ? rms_part_sum<4>(e, c, g * Q, Q) : Q <= 8 ? rms_part_sum<8>(e, c, g * Q, Q)
                                                                     : rms_part_sum<16>(e, c, g * Q, Q);
  red[g][t] = s;
  lds_barrier();
  if (threadIdx.x < MP) {
    float a = 0.f;
#pragma unroll
    for (int q = 0; q < G; ++q) a += red[q][threadIdx.x];
    rscale[threadIdx.x] = 1.0f / sqrtf(a * e.inv_d + e.eps);
  }
  lds_barrier();  // the scratch is free again
}

// ---- fused epilogue, bf16 path ----
// The accumulator fragment acc[nt][mt] of a lane holds features n .. n+3
// (n = (nb0 + nt) * 16 + 4 * (lane / 16)) of token t0 + mt * 16 + lane % 16.
// Operands that do not depend on the accumulators (the token's raster
// position, rotary factors, g_next, the old residual) are loaded first, in
// one batch, and the stores follow: no load waits behind a store.
__device__ __forceinline__ uint32_t pack2(uint16_t a, uint16_t b) { return (uint32_t)a | ((uint32_t)b << 16); }

// hi/lo bf16 planes of a pair: hi = bf16(x), lo = bf16(x - hi)
__device__ __forceinline__ void split2(float a, float b, uint32_t& hi, uint32_t& lo) {
  hi = cvt2bf(a, b);
  lo = cvt2bf(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xFFFF0000u));
}

template <int NT, int MT>
struct EpiOps {
  float4 a[NT][MT];  // RESID: old x[t][n..n+3]; QKV: (cos, sin) of rotary pairs j, j+1 at the token's position
  float4 g[NT];      // RESID: g_next[n..n+3]
  int pos[MT];       // QKV: raster position of the token
};

// block start f[b] of each fragment token (raw load; the position is formed at the epilogue)
template <int NT, int MT>
__device__ __forceinline__ void epi_block_starts(const EpiArgs& e, int M, int t0, int lane, EpiOps<NT, MT>& op) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int tl = mt * 16 + (lane & 15);
    op.pos[mt] = e.f[(t0 + (tl < M ? tl : M - 1)) / e.Kblk];
  }
}

// indexes are clamped into range (results of clamped lanes are never stored),
// so the loads carry no branches and issue back to back
template <int NT, int MT, class Mem = PlainMem>
__device__ __forceinline__ void epi_load(const EpiArgs& e, int nb0, int N, int M, int t0, int lane,
                                         EpiOps<NT, MT>& op) {
  const int nq = 4 * (lane >> 4);
  if (e.kind == EPI_RESID) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = (nb0 + nt) * 16 < N ? (nb0 + nt) * 16 + nq : nq;
      op.g[nt] = *(const float4*)(e.gnext + n);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int tl = mt * 16 + (lane & 15);
        op.a[nt][mt] = Mem::ldf4(e.x, ((size_t)(t0 + (tl < M ? tl : M - 1)) * e.ld + n) * 4);
      }
    }
  } else if (e.kind == EPI_QKV) {
    const int qN = e.Hq * e.D, half = e.D >> 1;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int tl = mt * 16 + (lane & 15);
      const int t = t0 + (tl < M ? tl : M - 1);
      op.pos[mt] += t % e.Kblk;
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = (nb0 + nt) * 16 + nq;
      const int nn = n < qN ? n : n - qN;
      const int j = (nn % e.D) >> 1;  // even: pairs j, j+1
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) op.a[nt][mt] = *(const float4*)(e.rope + (size_t)op.pos[mt] * half + j);
    }
  }
}

// returns per-mt partial sums of the new residual squared (RESID)
template <int NT, int MT, class Mem = PlainMem>
__device__ __forceinline__ void epi_store(const EpiArgs& e, const floatx4 (&acc)[NT][MT], const EpiOps<NT, MT>& op,
                                          int nb0, int N, int M, int t0, int lane, const float* rscale,
                                          float (&sq)[MT]) {
  const int nq = 4 * (lane >> 4);
  uint16_t* q = (uint16_t*)e.q;
  uint16_t* kc = (uint16_t*)e.kc;
  uint16_t* vc = (uint16_t*)e.vc;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int n = (nb0 + nt) * 16 + nq;
    if ((nb0 + nt) * 16 >= N) continue;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int tl = mt * 16 + (lane & 15);
      if (tl >= M) continue;
      const int t = t0 + tl;
      const float r = rscale[tl];
      const floatx4 v = acc[nt][mt];
      switch (e.kind) {
        case EPI_QKV: {
          const int b = t / e.Kblk, k = t - b * e.Kblk;
          const int pos = op.pos[mt];
          const int D = e.D, half = D >> 1;
          const int qN = e.Hq * D, kN = e.Hkv * D;
          if (n < qN + kN) {
            // features n..n+3 = rotary pairs (j, j + D/2) and (j + 1, j + 1 + D/2)
            const float4 cs = op.a[nt][mt];
            const float x0 = v[0] * r, y0 = v[1] * r, x1 = v[2] * r, y1 = v[3] * r;
            const float a0 = x0 * cs.x - y0 * cs.y, c0 = y0 * cs.x + x0 * cs.y;
            const float a1 = x1 * cs.z - y1 * cs.w, c1 = y1 * cs.z + x1 * cs.w;
            const bool isq = n < qN;
            const int nn = isq ? n : n - qN;
            const int head = nn / D, j = (nn - head * D) >> 1;  // j even: (j, j+1) share a tile lane
            if (isq) {
              // tiled q: rows r = (head within its KV group) * K + k of the KV head's block
              const int g = e.Hq / e.Hkv, hkv = head / g;
              const int r = (head - hkv * g) * e.Kblk + k;
              const size_t base = ((size_t)b * e.Hkv + hkv) * (size_t)e.qrows_pad * D;
              uint32_t h0, l0, h1, l1;
              split2(a0, a1, h0, l0);
              split2(c0, c1, h1, l1);
              const size_t i0 = base + tile16x32_index(r, j, D), i1 = base + tile16x32_index(r, j + half, D);
              Mem::st4(q, i0 * 2, h0);
              Mem::st4(q, i1 * 2, h1);
              Mem::st4(q, (e.q_plane + i0) * 2, l0);
              Mem::st4(q, (e.q_plane + i1) * 2, l1);
            } else {
              const size_t base = ((size_t)b * e.Hkv + head) * e.Lmax * D;
              Mem::st4(kc, (base + tile16x32_index(pos, j, D)) * 2, cvt2bf(a0, a1));
              Mem::st4(kc, (base + tile16x32_index(pos, j + half, D)) * 2, cvt2bf(c0, c1));
            }
          } else {
            const int nv = n - qN - kN;
            const int head = nv / D, dd = nv - head * D;
            const size_t base = ((size_t)b * e.Hkv + head) * (size_t)D * e.Lmax;
#pragma unroll
            for (int i = 0; i < 4; ++i) Mem::st2(vc, (base + vtile_index(dd + i, pos, e.Lmax)) * 2, f2bf(v[i] * r));
          }
          break;
        }
        case EPI_RESID: {
          const size_t i = (size_t)t * e.ld + n;
          const float4 xo = op.a[nt][mt];
          const float4 g = op.g[nt];
          const float4 xv = make_float4(xo.x + v[0], xo.y + v[1], xo.z + v[2], xo.w + v[3]);
          Mem::stf4(e.x, i * 4, xv);
          uint32_t h0, l0, h1, l1;
          split2(g.x * xv.x, g.y * xv.y, h0, l0);
          split2(g.z * xv.z, g.w * xv.w, h1, l1);
          Mem::st8(e.xn, i * 2, make_uint2(h0, h1));
          Mem::st8(e.xn, (e.xn_plane + i) * 2, make_uint2(l0, l1));
          sq[mt] += (xv.x * xv.x + xv.y * xv.y) + (xv.z * xv.z + xv.w * xv.w);
          break;
        }
        case EPI_SWIGLU: {
          // packed rows (2j, 2j+1) = (gate j, up j)
          const float g0 = v[0] * r, u0 = v[1] * r, g1 = v[2] * r, u1 = v[3] * r;
          const float s0 = g0 / (1.0f + expf(-g0)), s1 = g1 / (1.0f + expf(-g1));
          uint32_t hi, lo;
          split2(s0 * u0, s1 * u1, hi, lo);
          const size_t i = (size_t)t * e.ld + (n >> 1);
          Mem::st4(e.h, i * 2, hi);
          Mem::st4(e.h, (e.h_plane + i) * 2, lo);
          break;
        }
        default: {  // EPI_LOGITS
          Mem::stf4(e.logits, ((size_t)t * e.ld + n) * 4, make_float4(v[0] * r, v[1] * r, v[2] * r, v[3] * r));
          break;
        }
      }
    }
  }
}


// hi/lo bf16 planes of four consecutive fp32 values
template <class Mem = PlainMem>
__device__ __forceinline__ void store_split4(uint16_t* base, size_t i, size_t plane, floatx4 v) {
  uint2 w, x;
  split2(v[0], v[1], w.x, x.x);
  split2(v[2], v[3], w.y, x.y);
  Mem::st8(base, i * 2, w);
  Mem::st8(base, (i + plane) * 2, x);
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

template <int D, class Mem = PlainMem>
__device__ __forceinline__ void load_kv(KVTile<D>& t, const uint16_t* kbase, const uint16_t* vbase, int key0,
                                        int Lmax, int lane) {
  const int kb = key0 < Lmax - 32 ? key0 : Lmax - 32;
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int kd = 0; kd < D / 32; ++kd)
      t.k[kt][kd] = Mem::ld16(kbase, (((size_t)((kb >> 4) + kt) * (D / 32) + kd) * 512 + lane * 8) * 2);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt)
    t.v[dt] = Mem::ld16(vbase, (((size_t)dt * (Lmax >> 5) + (kb >> 5)) * 512 + lane * 8) * 2);
}

// max over lanes l, l ^ 16, l ^ 32 and l ^ 48 by gfx950's lane-swap
// instructions (VALU, no LDS round trip): permlane32_swap of v with itself
// leaves v[l] and v[l ^ 32] in the pair of every lane, permlane16_swap the
// same for l ^ 16
__device__ __forceinline__ float max_xor16_32(float v) {
  const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float m32 = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(m32), __float_as_uint(m32), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// lazy softmax reference (log2 units; probabilities stay within 2^8), and the
// reference before any visible key: finite, so that exp2(-inf - m) is 0, and
// below any score of the log2 domain
constexpr float AT_LAZY_LOG2 = 8.f;
constexpr float AT_M_NONE = -1e30f;

struct NoWait {
  __device__ __forceinline__ void operator()() const {}
};

// one 32-key block through the online softmax of the wave's query tiles
// QL: the query operands come from LDS (qs: tiles (qt, kd, plane) of 1 KiB in
// lane order) instead of registers (for callers short of registers).
// MASK = false: every key of the block is visible to every query (the block
// lies below the block's first position), so no causal mask is applied.
// The O rescale runs only when some lane's reference max moved (alpha != 1),
// and the reference moves only by more than AT_LAZY_LOG2: past the first
// blocks the accumulators stay untouched.
// after_scores: called once after the score MFMAs are issued (the V
// fragments' reads can start there, in the registers the K fragments held);
// before_pv: called once before the first PV product (a wait for them)
template <int D, int QPW, bool QL = false, bool MASK = true, class AfterS = NoWait, class BeforePV = NoWait>
__device__ __forceinline__ void attend_block(const KVTile<D>& t, int key0, const bf16x8 (&qh)[QPW][D / 32],
                                             const bf16x8 (&ql)[QPW][D / 32], const int (&qpos)[QPW],
                                             float scale_log2, int grp, float (&m)[QPW], float (&l)[QPW],
                                             floatx4 (&O)[QPW][D / 16], const uint16_t* qs = nullptr,
                                             int klim = 0x7fffffff, AfterS after_scores = AfterS{},
                                             BeforePV before_pv = BeforePV{}) {
  constexpr int KD = D / 32, DT = D / 16;
  floatx4 s[2][QPW];
  const uint16_t* qsl = qs + (threadIdx.x & 63) * 8;
  if constexpr (QL) asm volatile("" : "+v"(qsl));  // re-read every block (not hoisted into registers)
#pragma unroll
  for (int kt = 0; kt < 2; ++kt)
#pragma unroll
    for (int qt = 0; qt < QPW; ++qt) s[kt][qt] = floatx4{0.f, 0.f, 0.f, 0.f};
  // k steps and planes outermost: the 2 QPW accumulators take turns, so no
  // MFMA waits on the one just issued (each accumulator still sums kd = 0,
  // 1, ... with the hi plane before the lo plane)
#pragma unroll
  for (int kd = 0; kd < KD; ++kd)
#pragma unroll
    for (int pl = 0; pl < 2; ++pl)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int qt = 0; qt < QPW; ++qt) {
          const bf16x8 kf = __builtin_bit_cast(bf16x8, t.k[kt][kd]);
          bf16x8 a = pl ? ql[qt][kd] : qh[qt][kd];
          if constexpr (QL) {
            const uint16_t* p = qsl + ((size_t)(qt * KD + kd) * 2 + pl) * 512;
            a = __builtin_bit_cast(bf16x8, *(const u32x4*)p);
          }
          s[kt][qt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, a, s[kt][qt], 0, 0, 0);
        }
  after_scores();
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    float sv[8];              // raw scores (masked ones -inf)
    float tmax = -INFINITY;  // this lane's largest score of the block, then in log2 units
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int key = key0 + kt * 16 + 4 * grp + e;
        float v = s[kt][qt][e];
        if constexpr (MASK) v = (key <= qpos[qt] && key < klim) ? v : -INFINITY;
        sv[kt * 4 + e] = v;
        tmax = fmaxf(tmax, v);
      }
    tmax *= scale_log2;  // the scale is positive: the largest scaled score
    // The reference m moves only when a score exceeds it by more than
    // AT_LAZY_LOG2, so the probabilities lie in [0, 2^AT_LAZY_LOG2]; O and l
    // share the reference, so O / l is the same.  Each lane tests its own
    // scores: the row's maximum over its four lanes and the O rescale (a
    // read-modify-write of every accumulator) are needed only when some lane
    // of the wave exceeds -- at a chunk's first visible keys, then rarely.
    // m starts at AT_M_NONE, below any score: exp2 of (score - m) is then 0
    // for masked (-inf) scores, and the first visible score moves m.
    if (__builtin_amdgcn_ballot_w64(tmax > m[qt] + AT_LAZY_LOG2) != 0) {
      const float mx = max_xor16_32(tmax);
      const bool move = mx > m[qt] + AT_LAZY_LOG2;
      const float mnew = move ? mx : m[qt];
      const float alpha = __builtin_amdgcn_exp2f(m[qt] - mnew);  // 1 where m stays, 0 from AT_M_NONE
      l[qt] *= alpha;
      m[qt] = mnew;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) O[qt][dt] *= alpha;
    }
    float ps = 0.f;
    u32x4 pv, pw;  // hi / lo planes of the probabilities, pairs packed
#pragma unroll
    for (int i = 0; i < 8; i += 2) {
      // exponents are <= AT_LAZY_LOG2 (exp2 of -inf is 0): the hardware exp2 needs no range handling
      const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i], scale_log2, -m[qt]));
      const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i + 1], scale_log2, -m[qt]));
      ps += p0;
      ps += p1;
      uint32_t h, lo;
      split2(p0, p1, h, lo);
      pv[i / 2] = h;
      pw[i / 2] = lo;
    }
    l[qt] += ps;
    const bf16x8 pf = __builtin_bit_cast(bf16x8, pv);
    const bf16x8 pg = __builtin_bit_cast(bf16x8, pw);
    if (qt == 0) before_pv();
    // the hi plane into every accumulator, then the lo plane (each O tile
    // still takes hi before lo, and no MFMA waits on the one just issued)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      O[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, t.v[dt]), pf, O[qt][dt], 0, 0, 0);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      O[qt][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, t.v[dt]), pg, O[qt][dt], 0, 0, 0);
  }
}


constexpr int AT_KEYS = 32;        // keys per wave step
constexpr int AT_STEP = 128;       // chunk granularity in keys (one workgroup step)
constexpr int AT_MAX_CHUNKS = 64;
// query-split units stage K/V blocks in LDS: AT_KV_STAGES buffers of one
// 32-key block each (2 D/32 key tiles + D/16 value tiles of 1 KiB)
constexpr int AT_KV_STAGES = 4;
template <int D>
constexpr int at_kv_tiles() { return 2 * (D / 32) + D / 16; }
// four waves per workgroup (key-split units: one workgroup per CU, so a wave
// holds two K/V blocks, the one in use and the next, beside its queries and
// accumulators; query-split units: two workgroups per CU, K/V read from LDS)
template <int QPW>
struct AtShape {
  static constexpr int WAVES = 4;
  static constexpr int THREADS = WAVES * 64;
  static constexpr int STEP = WAVES * AT_KEYS;
};


// PF = 1: the next block's K/V tiles are loaded while the current one is used
// Attention for one work item of a launch: item = workgroup slot (single
// chunk: the query groups of one (sequence, KV head) share an XCD, they read
// the same K/V; several chunks: the chunks of one query group share an XCD,
// their partials meet in its L2).  Whole-workgroup call.  Returns the query
// group (sequence x KV head x query group index) whose output this workgroup
// wrote, or -1 (idle slot, or a chunk whose partial another workgroup merges).
// LDS: sm_o[NW*QPW*16*(D+4)], sm_m/sm_l[NW*QPW*16], is_last.
// Mem: queries, K/V and the output; PMem: the chunk partials; QL: queries
// staged in LDS (sm_q, QPW * D/32 * 2 KiB) instead of registers.
// QS: the waves split the query rows instead of the keys (a query group is
// NW * QPW * 16 rows, every wave streams every key block of the chunk from
// LDS (sm_kv; sm_o may share its bytes) and nothing is merged across waves):
// for query groups of many rows, whose K/V would otherwise be streamed once
// per 16-32 rows.
template <int D, int QPW, class Mem = PlainMem, bool PF = true, class PMem = PlainMem, bool QL = false,
          bool QS = false>
__device__ __forceinline__ int attn_unit(const AttnKArgs& a, int item, float* sm_o, float* sm_m, float* sm_l,
                                         int* is_last, uint16_t* sm_q = nullptr, uint16_t* sm_kv = nullptr) {
  static_assert(!(QS && QL), "query-split units keep the queries in registers");
  constexpr int NW = AtShape<QPW>::WAVES, NTH = AtShape<QPW>::THREADS;
  constexpr int STEP = QS ? AT_KEYS : AtShape<QPW>::STEP;  // keys between a wave's blocks
  constexpr int KD = D / 32;   // 32-wide k steps over the head dimension
  constexpr int DT = D / 16;   // 16-row d tiles of O^T
  constexpr int WROWS = QPW * 16;               // query rows of one wave
  constexpr int ROWS = QS ? NW * WROWS : WROWS;  // query rows of the workgroup
  constexpr int NWM = QS ? 1 : NW;               // waves merged per row
  constexpr int RS = D + 4;    // LDS row stride (floats): rows of one wave fall on different banks
  constexpr int NOUT = ROWS * D / 4;                          // float4 outputs of the workgroup
  constexpr int NV = (NOUT + NTH - 1) / NTH;    // per thread
  static_assert(2 * AT_MAX_CHUNKS * ROWS <= NW * WROWS * RS, "chunk statistics fit the O stage");
  // the workgroups of one (sequence, KV head) share an XCD: its query groups
  // read the same K/V
  int grp_id, c, z, qg;
  if (a.nchunk == 1) {
    xcd_unmap(item, a.nqg, a.xcd, z, qg);
    if (z >= a.heads) return -1;
    grp_id = z * a.nqg + qg;
    c = 0;
  } else {
    // every query group and key chunk of one (sequence, KV head) on one XCD:
    // the chunk partials meet in its L2, and the query groups' reads of the
    // same keys and values hit it (query groups of one chunk run together)
    int r;
    xcd_unmap(item, a.nqg * a.nchunk, a.xcd, z, r);
    if (z >= a.heads) return -1;
    c = r / a.nqg;
    qg = r - c * a.nqg;
    grp_id = z * a.nqg + qg;
  }
  const int b = z / a.Hkv, hkv = z - b * a.Hkv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int fb = a.f[b];
  const int ctx = fb + a.K;
  const int nch = (ctx + a.chunk - 1) / a.chunk;
  if (c >= nch) return -1;  // whole workgroup, before any barrier
  const int kbeg = c * a.chunk;
  const int kend = min(kbeg + a.chunk, ctx);
  const int rbase = qg * ROWS;

  const uint16_t* kbase = a.kc + ((size_t)b * a.Hkv + hkv) * a.Lmax * D;
  const uint16_t* vbase = a.vc + ((size_t)b * a.Hkv + hkv) * (size_t)D * a.Lmax;
  const int first = kbeg + (QS ? 0 : wave * AT_KEYS);
  const int nit = first < kend ? (kend - first + STEP - 1) / STEP : 0;
  const int wrbase = rbase + (QS ? wave * WROWS : 0);  // this wave's first query row

  // first K/V block in flight together with the queries.  K/V loads are never
  // conditional (a branch around loads makes the compiler wait for all of them
  // at the join): rows past the cache are clamped, and a block past the chunk
  // is loaded but never used.
  KVTile<D> ta, tb;
  if constexpr (!QS) load_kv<D, Mem>(ta, kbase, vbase, first, a.Lmax, lane);

  // query fragments (B operand of S^T = K Q^T): lane holds row col of tile qt, d = 8*grp.. (+32 kd);
  // q is fp32 carried as hi + lo bf16 operands
  bf16x8 qh[QPW][KD], ql[QPW][KD];
  int qpos[QPW];
  const uint16_t* qbase = a.q + (size_t)z * a.qrows_pad * D;
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    const int r = wrbase + qt * 16 + col;  // padded rows (r >= rows) exist and are masked
    qpos[qt] = r < a.rows ? fb + r % a.K : -1;
    // tiles past the padded rows (a 128-row query group ends past them) reload the last tile: masked rows
    const int tq = min((wrbase >> 4) + qt, (a.qrows_pad >> 4) - 1);
    const size_t qo = ((size_t)tq * KD) * 512 + lane * 8;
#pragma unroll
    for (int kd = 0; kd < KD; ++kd) {
      if constexpr (QL) {
        qh[qt][kd] = bf16x8{};
        ql[qt][kd] = bf16x8{};
      } else {
        qh[qt][kd] = __builtin_bit_cast(bf16x8, Mem::ld16(qbase, (qo + kd * 512) * 2));
        ql[qt][kd] = __builtin_bit_cast(bf16x8, Mem::ld16(qbase, (qo + a.q_plane + kd * 512) * 2));
      }
    }
  }
  if constexpr (QL) {
    // LDS DMA of the query tiles: tile i = (qt * KD + kd) * 2 + plane, 1 KiB each,
    // spread over the waves; every wave then reads all of them
    constexpr int NQ = QPW * KD * 2;
    constexpr int AUX = Mem::LDS_AUX;
    static_assert(NQ % NW == 0, "query tiles split evenly over the waves");
#pragma unroll
    for (int j = 0; j < NQ / NW; ++j) {
      const int i = wave * (NQ / NW) + j;
      const int qt = i / (2 * KD), kd = (i / 2) % KD, pl = i & 1;
      const uint16_t* src = qbase + ((size_t)((rbase >> 4) + qt) * KD + kd) * 512 + (pl ? a.q_plane : 0) + lane * 8;
      __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                       (void __attribute__((address_space(3)))*)(sm_q + (size_t)i * 512), 16, 0,
                                       AUX);
    }
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();
  }

  float m[QPW], l[QPW];
  floatx4 O[QPW][DT];
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    m[qt] = AT_M_NONE;
    l[qt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) O[qt][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  if constexpr (QS) {
    // long streams (query split): every wave needs every key block of the
    // chunk, so a block is copied once into LDS by LDS DMA (each wave copies
    // an equal share of its 1 KiB tiles, which the caches hold in MFMA operand
    // order) and all the waves read it from there; AT_KV_STAGES - 1 blocks
    // are in flight while one is multiplied, and no K/V data occupies
    // registers between blocks.  Blocks wholly below the frontier need no mask.
    constexpr int NT = at_kv_tiles<D>(), TPW = NT / NW, NST = AT_KV_STAGES;
    static_assert(NT % NW == 0 && TPW >= 1, "K/V tiles split evenly over the waves");
    const __amdgpu_buffer_rsrc_t krs = raw_rsrc(kbase), vrs = raw_rsrc(vbase);
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    auto issue = [&](int c) {
      const int key0 = first + c * STEP;
      const int kb = key0 < a.Lmax - AT_KEYS ? key0 : a.Lmax - AT_KEYS;  // rows past the cache: clamped, masked
      uint16_t* st = sm_kv + (size_t)(c % NST) * NT * 512;
#pragma unroll
      for (int j = 0; j < TPW; ++j) {
        const int i = wv * TPW + j;  // tile i: key tiles (kt, kd) first, then value tiles dt
        if (i < 2 * KD)
          dma16(krs, st + i * 512, lane * 16, (((kb >> 4) + i / KD) * KD + i % KD) * 1024);
        else
          dma16(vrs, st + i * 512, lane * 16, ((i - 2 * KD) * (a.Lmax >> 5) + (kb >> 5)) * 1024);
      }
    };
    const uint32_t kv0 = lds_addr(sm_kv) + lane * 16;
    auto attend = [&](int c, auto mask) {
      constexpr bool MASK = decltype(mask)::value;
      const uint32_t st = kv0 + (uint32_t)((c % NST) * NT * 1024);
      KVTile<D> t;
      u32x4(&kf)[2 * KD] = *reinterpret_cast<u32x4(*)[2 * KD]>(&t.k);
      ds_read_tiles<0>(kf, st, std::make_integer_sequence<int, 2 * KD>{});
      lgkm_wait<0>(kf);
      // the value tiles are read once the score MFMAs are issued, into the
      // registers the key tiles held: K and V are never live together
      auto read_v = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        ds_read_tiles<2 * KD>(t.v, st, std::make_integer_sequence<int, DT>{});
        __builtin_amdgcn_sched_barrier(0);  // the reads go out before the softmax
      };
      auto wait_v = [&]() {
        __builtin_amdgcn_sched_barrier(0);  // the softmax stays above the wait
        lgkm_wait<0>(t.v);
      };
      attend_block<D, QPW, false, MASK>(t, first + c * STEP, qh, ql, qpos, a.scale_log2, grp, m, l, O, nullptr,
                                        kend, read_v, wait_v);
    };
    auto step = [&](int c, auto mask) {
      // this wave's copies of block c are done (those of the up to NST - 2
      // later blocks already issued may not be)
      wait_vm_groups<TPW, NST - 2>(nit - 1 - c);
      // every wave's copies of block c are visible, and every wave is done with
      // block c - 1, whose buffer takes block c + NST - 1
      dma_barrier();
      if (c + NST - 1 < nit) issue(c + NST - 1);
      attend(c, mask);
    };
    // the blocks wholly below the frontier come first: one loop without the
    // mask, then the rest with it (two loops, not a branch per block, keep the
    // register assignment of each loop fixed)
    const int nfull = fb - first >= AT_KEYS ? min(nit, (fb - first - AT_KEYS) / STEP + 1) : 0;
    for (int c = 0; c < NST - 1 && c < nit; ++c) issue(c);
    for (int c = 0; c < nfull; ++c) step(c, std::false_type{});
    for (int c = nfull; c < nit; ++c) step(c, std::true_type{});
  } else if constexpr (PF) {
    // the next block is loaded before the current one is used and taken over
    // at the end of every iteration (an unconditional use: the compiler can
    // neither sink the loads past a loop exit nor drop the overlap)
    for (int it = 0; it < nit; ++it) {
      const int key0 = first + it * STEP;
      load_kv<D, Mem>(tb, kbase, vbase, key0 + STEP, a.Lmax, lane);
      if (key0 + AT_KEYS <= fb)
        attend_block<D, QPW, QL, false>(ta, key0, qh, ql, qpos, a.scale_log2, grp, m, l, O, sm_q);
      else
        attend_block<D, QPW, QL>(ta, key0, qh, ql, qpos, a.scale_log2, grp, m, l, O, sm_q);
      ta = tb;
    }
  } else {
    // one block in registers (for callers that keep other data live)
    for (int it = 0; it < nit; ++it) {
      const int key0 = first + it * STEP;
      attend_block<D, QPW, QL>(ta, key0, qh, ql, qpos, a.scale_log2, grp, m, l, O, sm_q);
      if (it + 1 < nit) load_kv<D, Mem>(ta, kbase, vbase, key0 + STEP, a.Lmax, lane);
    }
  }

  // stage this wave's triple: O^T accumulator element e of tile (qt, dt) is row
  // qt*16 + col, dims dt*16 + 4*grp + e
  if constexpr (QS) __syncthreads();  // every wave is done with the K/V stages sm_o may overlay
#pragma unroll
  for (int qt = 0; qt < QPW; ++qt) {
    l[qt] += __shfl_xor(l[qt], 16);
    l[qt] += __shfl_xor(l[qt], 32);
    float* row = sm_o + (size_t)(wave * WROWS + qt * 16 + col) * RS;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) *(floatx4*)(row + dt * 16 + 4 * grp) = O[qt][dt];
    if (grp == 0) {
      sm_m[wave * WROWS + qt * 16 + col] = m[qt];
      sm_l[wave * WROWS + qt * 16 + col] = l[qt];
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
    for (int w = 0; w < NWM; ++w) M = fmaxf(M, sm_m[w * ROWS + r]);
    float L = 0.f;
    floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < NWM; ++w) {
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
      const size_t oi = ((size_t)b * a.K + k) * (a.Hq * D) + (hkv * a.g + j) * D + 4 * d4;
      store_split4<Mem>(a.o, oi, a.o_plane, acc[i] * (1.f / Lr[i]));
    }
    return grp_id;
  }

  // publish the chunk's triple
  const size_t gbase = (size_t)grp_id * a.nchunk;
  {
    floatx4* Op = (floatx4*)(a.opart + (gbase + c) * ROWS * D);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = threadIdx.x + NTH * i;
      if (idx >= NOUT) continue;
      const floatx4 v = acc[i];
      PMem::stf4(Op, (size_t)idx * 16, make_float4(v[0], v[1], v[2], v[3]));
      const int r = idx / (D / 4), d4 = idx - r * (D / 4);
      if (d4 == 0) PMem::stf2(a.spart, ((gbase + c) * ROWS + r) * 8, make_float2(Mr[i], Lr[i]));
    }
  }
  // partial stores acknowledged by this XCD's L2, then count the arrival
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (!a.xcd) __threadfence();  // chunks on different XCDs: write back through L2
    unsigned prev = atomicAdd(&a.counters[grp_id], 1u);
    *is_last = (prev == (unsigned)(nch - 1));
    if (*is_last) a.counters[grp_id] = 0u;  // every chunk has arrived: re-arm for the next pass
    if (*is_last && !a.xcd) __threadfence();
  }
  __syncthreads();
  if (!*is_last) return -1;

  // last chunk: statistics of every (chunk, row) into LDS (parallel loads)
  float* cm = sm_o;                           // [nch][ROWS] chunk max
  float* cl = sm_o + AT_MAX_CHUNKS * ROWS;    // [nch][ROWS] chunk sum, then weight
  for (int i = threadIdx.x; i < nch * ROWS; i += NTH) {
    const float2 st = PMem::ldf2(a.spart, (gbase * ROWS + i) * 8);
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
  // weighted sum of the chunk partials in chunk order: a batch of a chunk's
  // loads is issued together, and only then weighted and summed (loads
  // interleaved with their uses were each waited for alone, one round trip
  // per load)
  const floatx4* G = (const floatx4*)(a.opart + gbase * ROWS * D);
  floatx4 v[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = floatx4{0.f, 0.f, 0.f, 0.f};
  constexpr int NB = NV < 8 ? NV : 8;  // loads in flight together (more spill registers here)
  static_assert(NV % NB == 0, "whole batches");
  for (int cc = 0; cc < nch; ++cc) {
#pragma unroll
    for (int i0 = 0; i0 < NV; i0 += NB) {
      float4 g4[NB];
      float wt[NB];
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int idx = threadIdx.x + NTH * (i0 + j);
        const int ic = idx < NOUT ? idx : NOUT - 1;
        g4[j] = PMem::ldf4(G, ((size_t)cc * NOUT + ic) * 16);
        wt[j] = cl[cc * ROWS + ic / (D / 4)];
      }
      __builtin_amdgcn_sched_barrier(0);  // the batch's loads and weight reads go out before their first use
#pragma unroll
      for (int j = 0; j < NB; ++j) v[i0 + j] += floatx4{g4[j].x, g4[j].y, g4[j].z, g4[j].w} * wt[j];
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
    const size_t oi = ((size_t)b * a.K + k) * (a.Hq * D) + (hkv * a.g + j) * D + 4 * d4;
    store_split4<Mem>(a.o, oi, a.o_plane, v[i] * (1.f / sm_l[r]));
  }
  return grp_id;
}

}  // namespace ssd
