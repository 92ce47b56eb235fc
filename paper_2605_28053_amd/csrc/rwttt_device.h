// Device-side number formats and vector access helpers shared by the kernel
// files.  Included inside namespace rwttt { namespace { ... } } of each file.
#pragma once

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ---------------------------------------------------------------------------
// Number formats
// ---------------------------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values -> packed bf16 pair (first in the low half), round to
// nearest even: one v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  const bf16x2_t h = __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t);
  return *reinterpret_cast<const uint32_t*>(&h);
}
__device__ __forceinline__ uint32_t bf16_rne(float f) { return bf16x2_rne(f, 0.f) & 0xffffu; }

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static float get(const void* p, size_t i) { return static_cast<const float*>(p)[i]; }
  __device__ static void put(void* p, size_t i, float v) { static_cast<float*>(p)[i] = v; }
};
template <> struct Elem<uint16_t> {
  __device__ static float get(const void* p, size_t i) {
    return __uint_as_float(uint32_t(static_cast<const uint16_t*>(p)[i]) << 16);
  }
  __device__ static void put(void* p, size_t i, float v) {
    static_cast<uint16_t*>(p)[i] = static_cast<uint16_t>(bf16_rne(v));
  }
};

// N consecutive elements at p as floats; p is 8-byte (N*2 == 8) or 16-byte aligned.
template <int N> __device__ __forceinline__ void load_n(const float* p, float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    const float4 t = *reinterpret_cast<const float4*>(p + i);
    v[i] = t.x; v[i + 1] = t.y; v[i + 2] = t.z; v[i + 3] = t.w;
  }
}
template <int N> __device__ __forceinline__ void load_n(const uint16_t* p, float (&v)[N]) {
  if constexpr (N == 8) {
    const uint4 t = *reinterpret_cast<const uint4*>(p);
    v[0] = bf16_lo(t.x); v[1] = bf16_hi(t.x); v[2] = bf16_lo(t.y); v[3] = bf16_hi(t.y);
    v[4] = bf16_lo(t.z); v[5] = bf16_hi(t.z); v[6] = bf16_lo(t.w); v[7] = bf16_hi(t.w);
  } else {
    static_assert(N == 4, "bf16 loads are 4 or 8 wide");
    const uint2 t = *reinterpret_cast<const uint2*>(p);
    v[0] = bf16_lo(t.x); v[1] = bf16_hi(t.x); v[2] = bf16_lo(t.y); v[3] = bf16_hi(t.y);
  }
}

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// NT: a streaming (non-temporal) store, for state that is not read again soon.
template <int N, bool NT = false>
__device__ __forceinline__ void store_n(float* p, const float (&v)[N]) {
#pragma unroll
  for (int i = 0; i < N; i += 4) {
    const f32x4_t t = {v[i], v[i + 1], v[i + 2], v[i + 3]};
    if (NT) __builtin_nontemporal_store(t, reinterpret_cast<f32x4_t*>(p + i));
    else *reinterpret_cast<f32x4_t*>(p + i) = t;
  }
}
template <int N, bool NT = false>
__device__ __forceinline__ void store_n(uint16_t* p, const float (&v)[N]) {
  static_assert(N == 4 || N == 8, "bf16 stores are 4 or 8 wide");
  if constexpr (N == 4) {
    const u32x2_t t = {bf16x2_rne(v[0], v[1]), bf16x2_rne(v[2], v[3])};
    if (NT) __builtin_nontemporal_store(t, reinterpret_cast<u32x2_t*>(p));
    else *reinterpret_cast<u32x2_t*>(p) = t;
  } else {
    const u32x4_t t = {bf16x2_rne(v[0], v[1]), bf16x2_rne(v[2], v[3]), bf16x2_rne(v[4], v[5]),
                       bf16x2_rne(v[6], v[7])};
    if (NT) __builtin_nontemporal_store(t, reinterpret_cast<u32x4_t*>(p));
    else *reinterpret_cast<u32x4_t*>(p) = t;
  }
}

// N elements of T held packed in 32-bit words, converted to fp32 on use.
template <typename T, int N> struct Packed {
  static constexpr int W = N * int(sizeof(T)) / 4;
  uint32_t w[W];
  __device__ __forceinline__ float get(int i) const {
    if constexpr (sizeof(T) == 4) return __uint_as_float(w[i]);
    else return (i & 1) ? __uint_as_float(w[i >> 1] & 0xffff0000u) : __uint_as_float(w[i >> 1] << 16);
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int i = 0; i < W; ++i) w[i] = 0u;
  }
};

template <bool NT, typename T, int N>
__device__ __forceinline__ void load_packed(const T* p, Packed<T, N>& r) {
  constexpr int W = Packed<T, N>::W;
  static_assert(W == 2 || W % 4 == 0, "8- or 16-byte multiples");
  if constexpr (W == 2) {
    const u32x2_t t = NT ? __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p))
                         : *reinterpret_cast<const u32x2_t*>(p);
    r.w[0] = t[0];
    r.w[1] = t[1];
  } else {
#pragma unroll
    for (int i = 0; i < W; i += 4) {
      const u32x4_t* q = reinterpret_cast<const u32x4_t*>(p) + i / 4;
      const u32x4_t t = NT ? __builtin_nontemporal_load(q) : *q;
      r.w[i] = t[0];
      r.w[i + 1] = t[1];
      r.w[i + 2] = t[2];
      r.w[i + 3] = t[3];
    }
  }
}
