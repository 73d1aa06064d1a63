// Device-side building blocks shared by the fused sub-kernels (gfx950).
//
//  * 128-bit global loads/stores of fp32 (4 per vector) and bf16 (8 per vector)
//  * exact bf16 -> fp32 widening, round-to-nearest-even fp32 -> bf16 narrowing
//    (v_cvt_pk_bf16_f32 on gfx950)
//  * wave64 all-reduce of arbitrary commutative combines: DPP quad
//    permutes and row mirrors inside 16 lanes, a ds_swizzle across the two
//    16-lane rows of each 32-lane half, and two readlanes across the halves
//  * LDS fold of per-wave partials for row groups wider than one wave
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

// Build-time tuning parameters (defaults measured on MI355X).  Streaming
// loads and stores use the non-temporal hint unless these are set to 0.
#ifndef FS_NT_LOAD
#define FS_NT_LOAD 1
#endif
#ifndef FS_NT_STORE
#define FS_NT_STORE 1
#endif

namespace fs {

constexpr bool kNtLoad = FS_NT_LOAD != 0;
constexpr bool kNtStore = FS_NT_STORE != 0;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// bf16 <-> fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 v;
  v.x = (__bf16)lo;
  v.y = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// ---------------------------------------------------------------------------
// element traits: storage type T <-> fp32, 16-byte vectors
// ---------------------------------------------------------------------------
template <typename T> struct Elem;

template <> struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ __forceinline__ static float load1(const float* p) { return *p; }
  __device__ __forceinline__ static void store1(float* p, float v) { *p = v; }
  __device__ __forceinline__ static void unpack(const u32x4& w, float* v) {
    v[0] = __uint_as_float(w.x); v[1] = __uint_as_float(w.y);
    v[2] = __uint_as_float(w.z); v[3] = __uint_as_float(w.w);
  }
  __device__ __forceinline__ static u32x4 pack(const float* v) {
    u32x4 w;
    w.x = __float_as_uint(v[0]); w.y = __float_as_uint(v[1]);
    w.z = __float_as_uint(v[2]); w.w = __float_as_uint(v[3]);
    return w;
  }
};

template <> struct Elem<uint16_t> {   // bf16 bit patterns
  static constexpr int kVec = 8;
  __device__ __forceinline__ static float load1(const uint16_t* p) { return bf16_to_f32(*p); }
  __device__ __forceinline__ static void store1(uint16_t* p, float v) { *p = f32_to_bf16(v); }
  __device__ __forceinline__ static void unpack(const u32x4& w, float* v) {
    v[0] = bf16_lo(w.x); v[1] = bf16_hi(w.x); v[2] = bf16_lo(w.y); v[3] = bf16_hi(w.y);
    v[4] = bf16_lo(w.z); v[5] = bf16_hi(w.z); v[6] = bf16_lo(w.w); v[7] = bf16_hi(w.w);
  }
  __device__ __forceinline__ static u32x4 pack(const float* v) {
    u32x4 w;
    w.x = pack_bf16x2(v[0], v[1]); w.y = pack_bf16x2(v[2], v[3]);
    w.z = pack_bf16x2(v[4], v[5]); w.w = pack_bf16x2(v[6], v[7]);
    return w;
  }
};

// A loaded element as fp32.  Loading the raw value and widening it where it
// is used keeps the wait for the load at the use, not at the load.
__device__ __forceinline__ float raw_f32(float v) { return v; }
__device__ __forceinline__ float raw_f32(uint16_t v) { return bf16_to_f32(v); }
// a byte-mask element: the additive value it stands for
__device__ __forceinline__ float raw_f32(uint8_t v) { return v != 0 ? -INFINITY : 0.f; }

// 128-bit loads/stores.  Streaming data is touched once, so it is loaded and
// stored non-temporally (it should not displace reused data from the caches);
// NT = true means "streaming", subject to the build-time switches above.
template <bool NT>
__device__ __forceinline__ u32x4 ld128(const void* p) {
  if constexpr (NT && kNtLoad) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  else return *reinterpret_cast<const u32x4*>(p);
}
template <bool NT>
__device__ __forceinline__ void st128(void* p, const u32x4& v) {
  if constexpr (NT && kNtStore) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
  else *reinterpret_cast<u32x4*>(p) = v;
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Load V consecutive elements of type T (one element, or 8, 16 or 32 bytes)
// as fp32.
template <typename T, int V, bool NT = true>
__device__ __forceinline__ void ldv(const T* p, float* out) {
  constexpr int kBytes = int(sizeof(T)) * V;
  constexpr int kPer16 = 16 / int(sizeof(T));
  if constexpr (V == 1) {
    out[0] = Elem<T>::load1(p);
  } else if constexpr (kBytes == 16) {
    Elem<T>::unpack(ld128<NT>(p), out);
  } else if constexpr (kBytes == 32) {
    Elem<T>::unpack(ld128<NT>(p), out);
    Elem<T>::unpack(ld128<NT>(p + kPer16), out + kPer16);
  } else if constexpr (kBytes == 8 && sizeof(T) == 2) {
    u32x2 w;
    if constexpr (NT && kNtLoad) w = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
    else w = *reinterpret_cast<const u32x2*>(p);
    out[0] = bf16_lo(w.x); out[1] = bf16_hi(w.x); out[2] = bf16_lo(w.y); out[3] = bf16_hi(w.y);
  } else {
    static_assert(kBytes == 16, "unsupported vector load width");
  }
}

// V consecutive elements of T held in registers exactly as loaded (bf16 stays
// packed two per dword until unpacked).  Loads are unconditional: callers
// clamp out-of-range addresses onto an in-bounds vector and mask the values
// afterwards, so the compiler can keep every load of a row in flight at once
// (a load under a per-lane branch forces a wait for all older loads).
// A byte mask (uint8_t) is held as loaded, four bytes per dword, and unpacks
// to the additive value it stands for: -inf where the byte is nonzero (an
// excluded position), 0 where it is zero.
template <typename T, int V>
struct Raw {
  static constexpr int kBytes = int(sizeof(T)) * V;
  static constexpr int kWords = V == 1 ? 1 : (kBytes + 3) / 4;
  uint32_t w[kWords];

  template <bool NT = true>
  __device__ __forceinline__ void load(const T* p) {
    if constexpr (sizeof(T) == 1) {
      static_assert(V == 1 || V == 4 || V == 8, "byte vectors of 1, 4 or 8");
      if constexpr (V == 1) {
        w[0] = *p;
      } else if constexpr (V == 4) {
        if constexpr (NT && kNtLoad) w[0] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
        else w[0] = *reinterpret_cast<const uint32_t*>(p);
      } else {
        u32x2 v;
        if constexpr (NT && kNtLoad) v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
        else v = *reinterpret_cast<const u32x2*>(p);
        w[0] = v.x; w[1] = v.y;
      }
    } else if constexpr (V == 1) {
      w[0] = __float_as_uint(Elem<T>::load1(p));
    } else if constexpr (kBytes == 16) {
      const u32x4 v = ld128<NT>(p);
      w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    } else if constexpr (kBytes == 32) {
      const u32x4 a = ld128<NT>(p), b = ld128<NT>(p + 16 / sizeof(T));
      w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
      w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
    } else {
      static_assert(kBytes == 8, "unsupported raw vector width");
      u32x2 v;
      if constexpr (NT && kNtLoad) v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
      else v = *reinterpret_cast<const u32x2*>(p);
      w[0] = v.x; w[1] = v.y;
    }
  }
  __device__ __forceinline__ void unpack(float* out) const {
    if constexpr (sizeof(T) == 1) {
#pragma unroll
      for (int i = 0; i < V; ++i)
        out[i] = ((w[i / 4] >> (8 * (i % 4))) & 0xffu) != 0u ? -INFINITY : 0.f;
    } else if constexpr (V == 1) {
      out[0] = __uint_as_float(w[0]);
    } else if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int i = 0; i < V; ++i) out[i] = __uint_as_float(w[i]);
    } else {
#pragma unroll
      for (int i = 0; i < V / 2; ++i) {
        out[2 * i] = bf16_lo(w[i]);
        out[2 * i + 1] = bf16_hi(w[i]);
      }
    }
  }
};

// Store V fp32 values as T (16 bytes when V > 1).
template <typename T, int V>
__device__ __forceinline__ void stv(T* p, const float* v) {
  if constexpr (V == 1) Elem<T>::store1(p, v[0]);
  else st128<true>(p, Elem<T>::pack(v));
}

// ---------------------------------------------------------------------------
// wave64 all-reduce
// ---------------------------------------------------------------------------
// DPP controls (GCN/CDNA encoding)
constexpr int kDppQuadSwap1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;  // lane i <-> 7-i within each 8
constexpr int kDppRowMirror = 0x140;      // lane i <-> 15-i within each 16

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
// ds_swizzle bit-mask mode: lane i reads lane (i ^ 16) within each 32 lanes
__device__ __forceinline__ float swizzle_xor16(float v) {
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (16 << 10)));
}
__device__ __forceinline__ float readlane(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// A partial result is a small struct P with static members
//   P::combine(const P&, const P&) -> P   (commutative, bit-symmetric)
//   P::template map<F>(const P&, F f)      applies f to every float field
// After wave_allreduce every lane holds the same combined value.
template <class P>
__device__ __forceinline__ P wave_allreduce(P p) {
  p = P::combine(p, P::map(p, [](float v) { return dpp<kDppQuadSwap1>(v); }));
  p = P::combine(p, P::map(p, [](float v) { return dpp<kDppQuadSwap2>(v); }));
  p = P::combine(p, P::map(p, [](float v) { return dpp<kDppRowHalfMirror>(v); }));
  p = P::combine(p, P::map(p, [](float v) { return dpp<kDppRowMirror>(v); }));
  p = P::combine(p, P::map(p, [](float v) { return swizzle_xor16(v); }));
  P a = P::map(p, [](float v) { return readlane(v, 0); });
  P b = P::map(p, [](float v) { return readlane(v, 32); });
  return P::combine(a, b);
}

// Row group of W waves: fold the per-wave results through LDS.  `lds` holds
// W partials; every thread returns the same value (folded in wave order).
template <int W, class P>
__device__ __forceinline__ P group_allreduce(P p, P* lds, int wave, int lane) {
  p = wave_allreduce(p);
  if constexpr (W == 1) {
    return p;
  } else {
    if (lane == 0) lds[wave] = p;
    __syncthreads();
    P acc = lds[0];
#pragma unroll
    for (int w = 1; w < W; ++w) acc = P::combine(acc, lds[w]);
    return acc;
  }
}

// ---------------------------------------------------------------------------
// activations
// ---------------------------------------------------------------------------
// GELU(z) = z * Phi(z) = max(z, 0) - |z| * Q(|z|), where Q(x) = erfc(x/sqrt 2)/2
// is the upper tail of the standard normal.  erfc(u) = (1 + a1 u + ... +
// a6 u^6)^-16 with the coefficients of Abramowitz & Stegun, Handbook of
// Mathematical Functions, formula 7.1.28 (|error of erf| <= 3e-7, u >= 0).
// The 1/sqrt(2) of the argument (a_i / 2^(i/2)) and the 1/2 of Q (2^(1/16)
// on the whole polynomial) are folded into the coefficients, so
// Q(x) = 1 / q(x)^16: six FMAs, four squarings, one v_rcp_f32 and two more
// operations, with no branch.  Large |z| overflow q^16 to +inf, giving Q = 0;
// |z| is clamped in the product so that GELU(+inf) = +inf.
__device__ __forceinline__ float gelu_erf(float z) {
  constexpr double k = 1.0442737824274138;       // 2^(1/16)
  constexpr double r2 = 1.4142135623730951;      // sqrt 2
  constexpr float c0 = float(k);
  constexpr float c1 = float(k * 0.0705230784 / r2);
  constexpr float c2 = float(k * 0.0422820123 / 2.0);
  constexpr float c3 = float(k * 0.0092705272 / (2.0 * r2));
  constexpr float c4 = float(k * 0.0001520143 / 4.0);
  constexpr float c5 = float(k * 0.0002765672 / (4.0 * r2));
  constexpr float c6 = float(k * 0.0000430638 / 8.0);
  const float x = fabsf(z);
  float q = fmaf(c6, x, c5);
  q = fmaf(q, x, c4);
  q = fmaf(q, x, c3);
  q = fmaf(q, x, c2);
  q = fmaf(q, x, c1);
  q = fmaf(q, x, c0);
  q = q * q;   // q^2
  q = q * q;   // q^4
  q = q * q;   // q^8
  q = q * q;   // q^16
  const float tail = __builtin_amdgcn_rcpf(q);     // Q(|z|)
  return fmaf(-fminf(x, 1e30f), tail, fmaxf(z, 0.f));
}

// logistic 1 / (1 + 2^(-z log2 e)): one v_exp_f32 and one v_rcp_f32
__device__ __forceinline__ float sigmoid(float z) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-z * kLog2e));
}

// R independent partials reduced together (one shuffle sequence for R rows)
template <class P, int R>
struct Multi {
  P p[R];
  __device__ __forceinline__ static Multi combine(const Multi& a, const Multi& b) {
    Multi o;
#pragma unroll
    for (int r = 0; r < R; ++r) o.p[r] = P::combine(a.p[r], b.p[r]);
    return o;
  }
  template <class F> __device__ __forceinline__ static Multi map(const Multi& a, F f) {
    Multi o;
#pragma unroll
    for (int r = 0; r < R; ++r) o.p[r] = P::map(a.p[r], f);
    return o;
  }
};

// plain sum
struct SumP {
  float s;
  __device__ __forceinline__ static SumP combine(const SumP& a, const SumP& b) { return {a.s + b.s}; }
  template <class F> __device__ __forceinline__ static SumP map(const SumP& a, F f) { return {f(a.s)}; }
};

}  // namespace fs
