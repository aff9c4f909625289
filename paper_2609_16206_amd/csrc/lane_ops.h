// Device helpers shared by the replica-simulation kernels: exact integer <->
// double conversions and collectives over aligned segments of S lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace rt {

constexpr double kTwo32 = 4294967296.0;
constexpr double kTwo52 = 4503599627370496.0;
// Simulated times stay below 2^52 ns (about 52 days): below it every time,
// sum and difference the kernels form is an exact integer in a double, and
// the double-to-int64 conversion below is exact.
constexpr double kTimeLimit = kTwo52;

// int64 -> double, exact for |x| < 2^53.
__device__ __forceinline__ double i64_to_f64(int64_t x) {
  return __builtin_fma((double)(int32_t)(x >> 32), kTwo32, (double)(uint32_t)(uint64_t)x);
}

// Integer-valued double in [0, 2^52) -> int64: adding 2^52 puts the integer
// in the low 52 bits of the significand (the exponent field is then fixed).
__device__ __forceinline__ int64_t f64_to_i64(double x) {
  const double y = x + kTwo52;
  const uint32_t hi = (uint32_t)__double2hiint(y) & 0xFFFFFu;
  return (int64_t)(((uint64_t)hi << 32) | (uint32_t)__double2loint(y));
}

// Maximum of two doubles that are never NaN, as one instruction (fmax first
// canonicalizes each operand it cannot prove canonical: one more
// instruction per operand).
__device__ __forceinline__ double max_f64(double a, double b) {
  double r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Hides a value's provenance from the optimizer (it stays in a VGPR), so that
// a select on it is not re-associated into a combination of lane masks.
template <typename T>
__device__ __forceinline__ T opaque(T x) {
  asm("" : "+v"(x));
  return x;
}

// Workgroup barrier for data exchanged through LDS: waits for this wave's
// LDS operations, then s_barrier.  Unlike __syncthreads it does not wait for
// the wave's global memory accesses (callers exchange nothing through global
// memory between waves), and the memory clobber keeps the compiler from
// moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Calls f(std::integral_constant<int, I>) for I = 0 .. N-1, so that code
// acting on register-resident slots under a branch indexes them with
// constants from the start (a loop index is constant only after unrolling,
// and the optimizer may turn such code into an access at a computed index
// first, which moves the slots to scratch memory).
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// ---------------------------------------------------------------------------
// Stores on a subset of a wave's lanes.  A vector store sends one L2 write
// request per active lane whatever its address (lanes that write one shared
// dummy slot are not merged), so a store made by one lane in eight through a
// dummy address costs as many requests as a full store.  These helpers switch
// exec to the lanes whose condition is nonzero for the store alone and
// restore it, inside one asm statement, so the compiler never sees exec
// change.  They keep five wait states after the vector compare that writes
// exec, and the exec restore after a 16-byte store is the wait state its data
// registers need before they may be rewritten.  Addresses must be valid on
// every lane all the same.
//
// The compiler does not count these stores in its memory-counter waits; a
// wait it places for a load issued before one of them therefore also waits
// for that store.  Callers issue them after the waits of their step.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void store_x4_if(uint32_t c, void* p, u32x4 v) {
  uint64_t sv;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "v_cmpx_ne_u32_e32 vcc, 0, %1\n\t"
      "s_nop 4\n\t"
      "global_store_dwordx4 %2, %3, off\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(sv)
      : "v"(c), "v"(p), "v"(v)
      : "vcc", "memory");
}

// 16 bytes at p and 4 bytes at q under one condition.
__device__ __forceinline__ void store_x4_b32_if(uint32_t c, void* p, u32x4 v, void* q, uint32_t w) {
  uint64_t sv;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "v_cmpx_ne_u32_e32 vcc, 0, %1\n\t"
      "s_nop 4\n\t"
      "global_store_dwordx4 %2, %3, off\n\t"
      "global_store_dword %4, %5, off\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(sv)
      : "v"(c), "v"(p), "v"(v), "v"(q), "v"(w)
      : "vcc", "memory");
}

// Two 4-byte and two 8-byte values (one simulated request's outcome).
__device__ __forceinline__ void store_out_if(uint32_t c, int32_t* p0, int32_t v0, int32_t* p1, int32_t v1, int64_t* p2,
                                             int64_t v2, int64_t* p3, int64_t v3) {
  uint64_t sv;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "v_cmpx_ne_u32_e32 vcc, 0, %1\n\t"
      "s_nop 4\n\t"
      "global_store_dword %2, %3, off\n\t"
      "global_store_dword %4, %5, off\n\t"
      "global_store_dwordx2 %6, %7, off\n\t"
      "global_store_dwordx2 %8, %9, off\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(sv)
      : "v"(c), "v"(p0), "v"(v0), "v"(p1), "v"(v1), "v"(p2), "v"(v2), "v"(p3), "v"(v3)
      : "vcc", "memory");
}

// ---------------------------------------------------------------------------
// Segment collectives over aligned groups of S lanes.  Within a 16-lane row:
// quad_perm xor 1, xor 2, then half-row mirror and row mirror (each step
// pairs every lane with one from the other half of its group, so after
// log2(S) steps every lane holds the group result).  Across rows, on the
// vector unit: v_permlane16_swap hands every lane of rows 0 and 1 (2 and 3)
// the other row's value, v_permlane32_swap every lane the other half's.  For
// S > 64 these reduce over the wave.
// ---------------------------------------------------------------------------
template <int C>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, C, 0xF, 0xF, true);
}

__device__ __forceinline__ uint32_t rl(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// Combines each lane's value with its paired row's (S >= 32) and half's
// (S >= 64), after the reduction within rows.
template <int S, typename Op>
__device__ __forceinline__ uint32_t cross_rows(uint32_t v, Op op) {
  if constexpr (S >= 32) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    v = op(r[0], r[1]);
  }
  if constexpr (S >= 64) {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    v = op(r[0], r[1]);
  }
  return v;
}

// Two independent segment minima, interleaved so that each DPP step of one
// fills the other's data-hazard wait.
template <int S>
__device__ __forceinline__ void seg_min2(uint32_t& v, uint32_t& w) {
  if constexpr (S >= 2) { v = min(v, dpp<0xB1>(v)); w = min(w, dpp<0xB1>(w)); }
  if constexpr (S >= 4) { v = min(v, dpp<0x4E>(v)); w = min(w, dpp<0x4E>(w)); }
  if constexpr (S >= 8) { v = min(v, dpp<0x141>(v)); w = min(w, dpp<0x141>(w)); }
  if constexpr (S >= 16) { v = min(v, dpp<0x140>(v)); w = min(w, dpp<0x140>(w)); }
  v = cross_rows<S>(v, [](uint32_t x, uint32_t y) { return min(x, y); });
  w = cross_rows<S>(w, [](uint32_t x, uint32_t y) { return min(x, y); });
}

template <int S>
__device__ __forceinline__ uint32_t seg_or(uint32_t v) {
  if constexpr (S >= 2) v |= dpp<0xB1>(v);
  if constexpr (S >= 4) v |= dpp<0x4E>(v);
  if constexpr (S >= 8) v |= dpp<0x141>(v);
  if constexpr (S >= 16) v |= dpp<0x140>(v);
  return cross_rows<S>(v, [](uint32_t x, uint32_t y) { return x | y; });
}

// Maximum over the whole wave of non-negative values.
__device__ __forceinline__ int32_t wave_max_nonneg(int32_t v) {
  uint32_t u = (uint32_t)v;
  u = max(u, dpp<0xB1>(u));
  u = max(u, dpp<0x4E>(u));
  u = max(u, dpp<0x141>(u));
  u = max(u, dpp<0x140>(u));
  u = max(max(rl(u, 0), rl(u, 16)), max(rl(u, 32), rl(u, 48)));
  return (int32_t)u;
}

// Two broadcasts at once: x from the lane of each segment where `ox` holds and
// y from the one where `oy` holds, the four halves reduced interleaved.
template <int S>
__device__ __forceinline__ void seg_bcast2_f64(double& x, bool ox, double& y, bool oy) {
  uint32_t a = ox ? (uint32_t)__double2loint(x) : 0u, b = ox ? (uint32_t)__double2hiint(x) : 0u;
  uint32_t c = oy ? (uint32_t)__double2loint(y) : 0u, d = oy ? (uint32_t)__double2hiint(y) : 0u;
  if constexpr (S >= 2) { a |= dpp<0xB1>(a); b |= dpp<0xB1>(b); c |= dpp<0xB1>(c); d |= dpp<0xB1>(d); }
  if constexpr (S >= 4) { a |= dpp<0x4E>(a); b |= dpp<0x4E>(b); c |= dpp<0x4E>(c); d |= dpp<0x4E>(d); }
  if constexpr (S >= 8) { a |= dpp<0x141>(a); b |= dpp<0x141>(b); c |= dpp<0x141>(c); d |= dpp<0x141>(d); }
  if constexpr (S >= 16) { a |= dpp<0x140>(a); b |= dpp<0x140>(b); c |= dpp<0x140>(c); d |= dpp<0x140>(d); }
  const auto orf = [](uint32_t x, uint32_t y) { return x | y; };
  a = cross_rows<S>(a, orf);
  b = cross_rows<S>(b, orf);
  c = cross_rows<S>(c, orf);
  d = cross_rows<S>(d, orf);
  x = __hiloint2double((int)b, (int)a);
  y = __hiloint2double((int)d, (int)c);
}

// Values of two lanes of each segment, read by every lane of it: x from
// segment lane lx and y from segment lane ly (each in [0, S)), one
// ds_bpermute per 32-bit half (no memory access: the lanes exchange through
// the LDS crossbar).
template <int S>
__device__ __forceinline__ void seg_pick2_f64(double& x, int32_t lx, double& y, int32_t ly, int lane) {
  const int base = lane & ~(S - 1);
  const int ax = (base + lx) << 2, ay = (base + ly) << 2;
  const int xl = __builtin_amdgcn_ds_bpermute(ax, __double2loint(x));
  const int xh = __builtin_amdgcn_ds_bpermute(ax, __double2hiint(x));
  const int yl = __builtin_amdgcn_ds_bpermute(ay, __double2loint(y));
  const int yh = __builtin_amdgcn_ds_bpermute(ay, __double2hiint(y));
  x = __hiloint2double(xh, xl);
  y = __hiloint2double(yh, yl);
}

// A 32-bit value of segment lane lv, read by every lane of the segment.
template <int S>
__device__ __forceinline__ int32_t seg_pick(int32_t v, int32_t lv, int lane) {
  return __builtin_amdgcn_ds_bpermute(((lane & ~(S - 1)) + lv) << 2, v);
}

// Lowest lane (relative to the segment, or to the wave for S >= 64) of each
// segment where `pred` holds; -1 where it holds nowhere.
template <int S>
__device__ __forceinline__ int32_t seg_first(bool pred, int lane) {
  const uint64_t b = __ballot(pred);
  if constexpr (S >= 64) {
    return __ffsll((unsigned long long)b) - 1;
  } else {
    const uint32_t half = lane < 32 ? (uint32_t)b : (uint32_t)(b >> 32);
    const int sh = (lane & 31) & ~(S - 1);
    const uint32_t mask = (S == 32) ? 0xffffffffu : ((1u << (S & 31)) - 1u);
    return __ffs((half >> sh) & mask) - 1;
  }
}

}  // namespace rt
