// device_common.hpp -- device helpers shared by the HIP kernels of libar.so:
// wave/tile constants, 16-byte and 4-byte loads/stores (optionally
// nontemporal), the combination function and the precomputed division.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "ar_internal.hpp"

namespace ar {

constexpr int kWave = 64;
constexpr int kBlock = 256;                 // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int64_t kTile = int64_t(kWave) * 4;  // elements per wave tile: one 16-byte vector per lane
constexpr int64_t kMaxGrid = int64_t(1) << 22; // workgroups per launch; beyond it waves loop

template <typename T>
struct alignas(16) V4 {
  T v[4];
};

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
template <typename T> struct Ext;
template <> struct Ext<float> { using type = f32x4; };
template <> struct Ext<int32_t> { using type = i32x4; };

// 16-byte load/store; NT marks them nontemporal (streamed past the caches),
// which pays for launches far larger than the 256 MB Infinity Cache.
template <bool NT, typename T>
__device__ __forceinline__ V4<T> ld4(const V4<T>* p) {
  if constexpr (NT) {
    using E = typename Ext<T>::type;
    const E e = __builtin_nontemporal_load(reinterpret_cast<const E*>(p));
    V4<T> r;
    r.v[0] = e[0]; r.v[1] = e[1]; r.v[2] = e[2]; r.v[3] = e[3];
    return r;
  } else {
    return *p;
  }
}

template <bool NT, typename T>
__device__ __forceinline__ void st4(V4<T>* p, const V4<T>& v) {
  if constexpr (NT) {
    using E = typename Ext<T>::type;
    E e;
    e[0] = v.v[0]; e[1] = v.v[1]; e[2] = v.v[2]; e[3] = v.v[3];
    __builtin_nontemporal_store(e, reinterpret_cast<E*>(p));
  } else {
    *p = v;
  }
}

template <int OP>
__device__ __forceinline__ float comb(float a, float b) {
  if constexpr (OP == 0) return a + b;
  else return b > a ? b : a;
}

template <int OP>
__device__ __forceinline__ int32_t comb(int32_t a, int32_t b) {
  if constexpr (OP == 0) return int32_t(uint32_t(a) + uint32_t(b));
  else return b > a ? b : a;
}

// 4-byte load/store, optionally nontemporal.
template <bool NT, typename T>
__device__ __forceinline__ T ld1(const T* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT, typename T>
__device__ __forceinline__ void st1(T* p, T v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

template <int OP, typename T>
__device__ __forceinline__ V4<T> comb4(const V4<T>& a, const V4<T>& b) {
  V4<T> r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r.v[i] = comb<OP>(a.v[i], b.v[i]);
  return r;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv& f) {
  if (f.l == 0) return n;
  const uint32_t t = __umulhi(n, f.m);
  return (t + ((n - t) >> 1)) >> (f.l - 1);
}

// The column that one lane of wave tile t works on in a block-tiled column
// launch: sets the block b (the same for the whole wave, so the rank
// rotation and its pointers stay uniform) and the element index e of the
// column in every rank buffer; returns whether the lane holds a column.
//
// Blocked tiles (a.packed = 0): t = (instance * P + block) * tiles + tile,
// 64 columns of one block per tile, the tiles of a block laid on 256-byte
// boundaries of its root rank's buffer (its first and last tile partial).
// Packed tiles (a.packed = 1, blocks of at most 64 elements): t = group * P
// + block, and the tile covers that block in a.ipw consecutive instances,
// lane j * maxlen + c holding column c of instance group * ipw + j, so short
// blocks fill the wave; the four waves of a workgroup take neighbouring
// blocks of the same instances.
__device__ __forceinline__ bool col_tile_column(const ColArgs& a, uint32_t t, int lane, int32_t& b, int64_t& e) {
  if (a.packed) {
    const uint32_t g = fdiv(t, a.pdiv);
    b = int32_t(t - g * a.pdiv.d);
    const uint32_t j = fdiv(uint32_t(lane), a.lendiv);
    const int64_t c = int64_t(lane) - int64_t(j) * a.lendiv.d;
    const uint32_t inst = g * a.ipw + j;
    e = int64_t(inst) * a.stride + int64_t(b) * a.q + (b < a.m ? b : a.m) + c;
    return j < a.ipw && inst < a.batch && c < a.q + (b < a.m ? 1 : 0);
  }
  const uint32_t seg = fdiv(t, a.tiles);  // seg = instance * P + block
  const uint32_t tile = t - seg * a.tiles.d;
  const uint32_t inst = fdiv(seg, a.pdiv);
  b = int32_t(seg - inst * a.pdiv.d);
  const int64_t len = a.q + (b < a.m ? 1 : 0);
  const int64_t e0 = int64_t(inst) * a.stride + int64_t(b) * a.q + (b < a.m ? b : a.m);
  const int64_t lo = ((reinterpret_cast<uintptr_t>(a.user[b]) >> 2) + e0) & (kWave - 1);
  const int64_t c = int64_t(tile) * kWave - lo + lane;
  e = e0 + c;
  return c >= 0 && c < len;
}

}  // namespace ar
