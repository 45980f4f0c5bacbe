// Device prelude included by every generated gfx950 kernel.
//
// Storage dtypes are fp32, fp16 (_Float16) and bf16 (__bf16); all arithmetic
// is fp32 in registers.  Conversions to fp16 / bf16 round to nearest even.
#pragma once

typedef long long i64;
typedef _Float16 f16;
typedef __bf16 bf16;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

struct KArgs {
  void* p[KORCH_NARGS];
};

// Half-precision MFMA B-operand fragment from an LDS tile stored [k][n] (n
// contiguous, row pitch `pitch` elements).  Each lane passes the address of
// row k0 + (lane%16)/4, column n0 + 4*(lane%4); the transposing read returns
// to lane i of every 16-lane group the 4 elements (k0..k0+3, n0 + i); a second
// read 4 rows below completes the 8 consecutive k of the fragment.
__device__ __forceinline__ s16x8 lds_tr_k8(const void* p, int pitch) {
  typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
  s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
  s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)((const short*)p + 4 * pitch));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// ---- scalar conversions ----------------------------------------------------
__device__ __forceinline__ float tof(float x) { return x; }
__device__ __forceinline__ float tof(f16 x) { return (float)x; }
__device__ __forceinline__ float tof(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T fromf(float x);
template <> __device__ __forceinline__ float fromf<float>(float x) { return x; }
template <> __device__ __forceinline__ f16 fromf<f16>(float x) { return (f16)x; }
template <> __device__ __forceinline__ bf16 fromf<bf16>(float x) { return (bf16)x; }

// ---- vector loads / stores of V consecutive elements (16-B aligned when V*size == 16)
template <int V, typename T> struct VecOf {
  typedef T type __attribute__((ext_vector_type(V)));
};
template <typename T> struct VecOf<1, T> {
  typedef T type;
};

template <int V, typename T> using vec_t = typename VecOf<V, T>::type;

template <int V, typename T>
__device__ __forceinline__ void ldv(float* d, const T* __restrict__ p) {
  if constexpr (V == 1) {
    d[0] = tof(*p);
  } else {
    typedef typename VecOf<V, T>::type VT;
    VT v = *reinterpret_cast<const VT*>(p);
#pragma unroll
    for (int i = 0; i < V; ++i) d[i] = tof(v[i]);
  }
}

template <int V, typename T>
__device__ __forceinline__ void stv(T* __restrict__ p, const float* s) {
  if constexpr (V == 1) {
    *p = fromf<T>(s[0]);
  } else {
    typedef typename VecOf<V, T>::type VT;
    VT v;
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = fromf<T>(s[i]);
    *reinterpret_cast<VT*>(p) = v;
  }
}

template <typename T> __device__ __forceinline__ float ld1(const T* __restrict__ p) { return tof(*p); }
template <typename T> __device__ __forceinline__ void st1(T* __restrict__ p, float v) { *p = fromf<T>(v); }

// ---- kernel output stores --------------------------------------------------
// A kernel output is written once and read only by later kernels.  It is
// stored with the device-scope cache policy (sc1), which writes it through
// the XCD's L2 to the device's point of coherence while the kernel runs.  A
// plain store leaves the line dirty in L2, and the release at the end of the
// kernel then writes back every such line after the last workgroup has
// finished (about 0.16 us per MB of output on this part, not overlapped with
// any work).  `base` is the tensor's (uniform) base pointer, `off` the element
// offset of the first of V consecutive elements; tensors stay below 2 GiB.
typedef unsigned int u32x2_ __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4o_ __attribute__((ext_vector_type(4)));
template <int V, typename T>
__device__ __forceinline__ void stv_out(T* base, i64 off, const float* s) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7fffffff, 0x00020000);
  const unsigned o = (unsigned)(off * (i64)sizeof(T));
  typedef typename VecOf<V, T>::type VT;
  VT v;
  if constexpr (V == 1) {
    v = fromf<T>(s[0]);
  } else {
#pragma unroll
    for (int i = 0; i < V; ++i) v[i] = fromf<T>(s[i]);
  }
  constexpr int B = V * (int)sizeof(T);
  if constexpr (B == 16) {
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4o_, v), r, o, 0, 16);
  } else if constexpr (B == 8) {
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_, v), r, o, 0, 16);
  } else if constexpr (B == 4) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, o, 0, 16);
  } else if constexpr (B == 2) {
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, v), r, o, 0, 16);
  } else if constexpr (B % 16 == 0) {
    struct W {
      u32x4o_ q[B / 16];
    };
    const W w = __builtin_bit_cast(W, v);
#pragma unroll
    for (int q = 0; q < B / 16; ++q) __builtin_amdgcn_raw_buffer_store_b128(w.q[q], r, o + 16 * q, 0, 16);
  } else {
    *reinterpret_cast<VT*>(base + off) = v;
  }
}
// 16 bytes already in the storage dtype, at byte offset `boff` of a kernel
// output, with the same write-through policy.
__device__ __forceinline__ void st16_out(void* base, i64 boff, uint4 v) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(base, 0, 0x7fffffff, 0x00020000);
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4o_, v), r, (unsigned)boff, 0, 16);
}
// ---- loads that read zero where a condition fails, without a branch ------
// A guarded load (`if (ok) x = *p;`) becomes a branch around the load, and the
// compiler waits for every load in flight where the branches join.  A buffer
// load whose offset is out of range returns zero instead, so these loads are
// issued back to back.  `boff` is a byte offset from `base` (tensors below 2 GiB).
__device__ __forceinline__ uint4 ld16_or_zero(const void* base, i64 boff, bool ok) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, 0x00020000);
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, ok ? (unsigned)boff : 0x80000000u, 0, 0));
}
__device__ __forceinline__ float ld4f_or_zero(const float* base, i64 eoff, bool ok) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, 0x7fffffff, 0x00020000);
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, ok ? (unsigned)(eoff * 4) : 0x80000000u, 0, 0));
}
// V consecutive elements at element offset `off` of `base` into fp32
// registers, zeros where `ok` is false, without a branch (V * sizeof(T) of 4,
// 8 or 16 bytes; tensors below 2 GiB).
template <int V, typename T>
__device__ __forceinline__ void ldv_or_zero(float* d, const T* base, i64 off, bool ok) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(base), 0, 0x7fffffff, 0x00020000);
  const unsigned o = ok ? (unsigned)(off * (i64)sizeof(T)) : 0x80000000u;
  typedef typename VecOf<V, T>::type VT;
  constexpr int B = V * (int)sizeof(T);
  static_assert(V > 1 && (B == 4 || B == 8 || B == 16), "ldv_or_zero: 4, 8 or 16 bytes of two or more elements");
  VT v;
  if constexpr (B == 16) {
    v = __builtin_bit_cast(VT, __builtin_amdgcn_raw_buffer_load_b128(r, o, 0, 0));
  } else if constexpr (B == 8) {
    v = __builtin_bit_cast(VT, __builtin_amdgcn_raw_buffer_load_b64(r, o, 0, 0));
  } else {
    v = __builtin_bit_cast(VT, __builtin_amdgcn_raw_buffer_load_b32(r, o, 0, 0));
  }
#pragma unroll
  for (int i = 0; i < V; ++i) d[i] = tof(v[i]);
}
// One element at element offset `off` of `base` as fp32, zero where `ok` is
// false, without a branch (tensors below 2 GiB).
template <typename T> __device__ __forceinline__ float ld1_or_zero(const T* base, i64 off, bool ok) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(base), 0, 0x7fffffff, 0x00020000);
  const unsigned o = ok ? (unsigned)(off * (i64)sizeof(T)) : 0x80000000u;
  if constexpr (sizeof(T) == 4) {
    return tof(__builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(r, o, 0, 0)));
  } else {
    static_assert(sizeof(T) == 2, "ld1_or_zero: 2- or 4-byte elements");
    return tof(__builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b16(r, o, 0, 0)));
  }
}
template <typename T> __device__ __forceinline__ void st1_out(T* base, i64 off, float v) {
  stv_out<1, T>(base, off, &v);
}

// ---- elementwise functions (fp32) -----------------------------------------
// max / min / ReLU are the single-instruction v_max_f32 / v_min_f32 (a
// compare and a select would take two, with the compare's mask in scalar
// registers); they agree with the comparison forms on every non-NaN input
// (up to the sign of a zero result).
__device__ __forceinline__ float k_relu(float x) { return __builtin_fmaxf(x, 0.0f); }
__device__ __forceinline__ float k_rsqrt(float x) { return 1.0f / sqrtf(x); }
__device__ __forceinline__ float k_gelu_tanh(float x) {
  // 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))
  const float c = 0.7978845608028654f;
  return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}
__device__ __forceinline__ float k_max(float a, float b) { return __builtin_fmaxf(a, b); }
__device__ __forceinline__ float k_min(float a, float b) { return __builtin_fminf(a, b); }

// Mish written as x * n / (n + 2) with n = e^x (e^x + 2), which equals
// x * tanh(log(1 + e^x)) exactly.  For x >= 20 the quotient rounds to 1 in
// fp32, so the exponent's argument is clamped there (no overflow, no branch).
__device__ __forceinline__ float k_mish(float x) {
  float ex = expf(k_min(x, 20.0f));
  float n = ex * (ex + 2.0f);
  return x * (n / (n + 2.0f));
}

// Fast variants for kernels whose results are stored in fp16 / bf16: the
// hardware exp2 / log2 / reciprocal approximations (a few ulp of fp32),
// far below the 2^-11 / 2^-8 spacing of the stored values.
__device__ __forceinline__ float f_exp(float x) { return __expf(x); }
__device__ __forceinline__ float f_log(float x) { return __logf(x); }
__device__ __forceinline__ float f_div(float x, float y) { return x * __builtin_amdgcn_rcpf(y); }
// tanh(x) = 1 - 2 / (e^{2x} + 1): saturates to +-1 when e^{2x} overflows or vanishes.
__device__ __forceinline__ float f_tanh(float x) { return 1.0f - f_div(2.0f, f_exp(2.0f * x) + 1.0f); }
__device__ __forceinline__ float f_rsqrt(float x) { return __builtin_amdgcn_rsqf(x); }
// 0.5 x (1 + tanh(u)) equals x / (1 + e^{-2u}) exactly; with
// u = sqrt(2/pi) (x + 0.044715 x^3) that is one base-2 exponential of
// -2 sqrt(2/pi) / ln(2) * x (1 + 0.044715 x^2) and one reciprocal.  Large |x|
// saturate to x and -0.
__device__ __forceinline__ float f_gelu_tanh(float x) {
  // k x (1 + 0.044715 x^2) = x * fma(x^2, 0.044715 k, k): five VALU operations
  // and two transcendentals per element
  const float k = -2.302208198144325f;
  const float t = x * __builtin_fmaf(x * x, 0.044715f * k, k);
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
}
__device__ __forceinline__ float f_mish(float x) {
  float ex = f_exp(k_min(x, 20.0f));
  float n = ex * (ex + 2.0f);
  return x * f_div(n, n + 2.0f);
}

// ---- fp32 partial results handed from workgroup to workgroup --------------
// Device-scope (agent) atomic stores and loads are performed at the point of
// coherence of the whole device, so a value one workgroup stores this way is
// read by a workgroup on another XCD without an L2 write-back on the writer's
// side or an L2 invalidate on the reader's (the device-scope release and
// acquire fences would do both for the whole L2).
__device__ __forceinline__ void coherent_store(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float coherent_load(float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Four consecutive fp32 partials at byte offset `off` of a buffer (16-byte
// aligned), loaded or stored with the cache policy of the device-scope
// accesses above (performed at the device's point of coherence).
__device__ __forceinline__ float4 coherent_load4(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16));
}
typedef unsigned int u32x4_ __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void coherent_store4(__amdgpu_buffer_rsrc_t r, unsigned off, float4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_, v), r, off, 0, 16);
}

// ---- reductions across a group of G lanes of a wavefront (G power of two <= 64)
template <int G> __device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int m = G / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
template <int G> __device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int m = G / 2; m >= 1; m >>= 1) v = k_max(v, __shfl_xor(v, m, 64));
  return v;
}
