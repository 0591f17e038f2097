// emul_wave.h - single-lane host stand-ins for the wave intrinsics used by
// paper_2601_18999_amd/csrc/kvr_core.h, so its logic can be compiled with g++
// and replayed on the CPU in tests (KVR_WAVE = 1: every lane-parallel loop
// becomes a sequential loop, every ballot has one lane).  Test-only.
#pragma once
#include <cstdint>
#include <cstddef>

#define KVR_WAVE 1
#define __device__
#define __forceinline__ inline
#define __noinline__ __attribute__((noinline))
#define __builtin_amdgcn_wave_barrier() ((void)0)
#define __builtin_amdgcn_fence(order, scope) ((void)0)

struct kvr_emul_dim3 { unsigned x, y, z; };
static const kvr_emul_dim3 threadIdx = {0, 0, 0};
struct int2 { int x, y; };
struct alignas(16) int4 { int x, y, z, w; };

inline uint64_t __ballot(bool p) { return p ? 1ull : 0ull; }
inline int __shfl(int v, int, int) { return v; }
inline int __builtin_amdgcn_readlane(int v, int) { return v; }
// one lane: every DPP source lies outside the row, so the lane keeps its value
inline int __builtin_amdgcn_update_dpp(int old, int, int, int, int, bool) { return old; }
inline int __builtin_amdgcn_readfirstlane(int v) { return v; }
inline void __builtin_amdgcn_s_sleep(int) {}
inline long long wall_clock64() { return 0; }
#define __ATOMIC_ACQUIRE_EMUL 0
template <typename T> inline T __hip_atomic_load(const T* p, int, int) { return *p; }
template <typename T> inline void __hip_atomic_store(T* p, T v, int, int) { *p = v; }
template <typename T> inline T __hip_atomic_fetch_add(T* p, T v, int, int) { T o = *p; *p += v; return o; }
#ifndef __HIP_MEMORY_SCOPE_WORKGROUP
#define __HIP_MEMORY_SCOPE_WORKGROUP 3
#endif
inline int atomicSub(int* p, int v) { int o = *p; *p -= v; return o; }
inline int atomicAdd(int* p, int v) { int o = *p; *p += v; return o; }
inline int __shfl_xor(int v, int, int) { return v; }
inline int __shfl_up(int v, int, int) { return v; }
inline int __ffsll(unsigned long long m) { return __builtin_ffsll((long long)m); }
inline int __popcll(unsigned long long m) { return __builtin_popcountll(m); }
inline int __clzll(long long m) { return m ? __builtin_clzll((unsigned long long)m) : 64; }
inline uint64_t __umul64hi(uint64_t a, uint64_t b) {
  return (uint64_t)(((unsigned __int128)a * b) >> 64);
}
