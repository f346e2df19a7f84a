// Device helpers for the SAKI gfx950 kernels: vector loads of logit rows,
// wave/block reductions, Philox-4x32-10 and bf16 conversion.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace saki {

constexpr int WAVE = 64;
constexpr int CHUNK = 1024;            // vocab entries per race chunk; one wave tile
constexpr int EPL = CHUNK / WAVE;      // 16 entries per lane per chunk
constexpr int MAX_VOCAB = 1 << 21;
constexpr int MAX_CHUNKS = MAX_VOCAB / CHUNK;

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr double LN2_D = 0.6931471805599453094;

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float flog2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float finf() { return __builtin_huge_valf(); }
// Three-input maximum / minimum (v_max3_f32 / v_min3_f32) applied to the
// operands as they are: fmaxf on values unpacked from bf16 bits first quiets
// each operand (one more instruction per entry), which a row statistic does
// not need (a NaN entry makes the row non-finite either way).
__device__ __forceinline__ float max3_raw(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float min3_raw(float a, float b, float c) {
  float r;
  asm("v_min3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}

// ---------------------------------------------------------------------------
// Row element layout inside a chunk.  Lane l of the wave that owns chunk c
// holds entries c*1024 + 8l + e (e < 8) and c*1024 + 512 + 8l + (e - 8)
// (e >= 8): two fully coalesced 1 KiB (bf16) segments per array.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int elem_offset(int lane, int e) {
  return (e < 8) ? (8 * lane + e) : (512 + 8 * lane + (e - 8));
}

template <typename T>
struct Loader;

template <>
struct Loader<uint16_t> {  // bf16 stored as raw 16-bit words
  static __device__ __forceinline__ void load8(const uint16_t* p, float* x) {
    const uint4 q = *reinterpret_cast<const uint4*>(p);
    x[0] = __uint_as_float(q.x << 16);
    x[1] = __uint_as_float(q.x & 0xffff0000u);
    x[2] = __uint_as_float(q.y << 16);
    x[3] = __uint_as_float(q.y & 0xffff0000u);
    x[4] = __uint_as_float(q.z << 16);
    x[5] = __uint_as_float(q.z & 0xffff0000u);
    x[6] = __uint_as_float(q.w << 16);
    x[7] = __uint_as_float(q.w & 0xffff0000u);
  }
  static __device__ __forceinline__ float load1(const uint16_t* p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
  }
};

template <>
struct Loader<float> {
  static __device__ __forceinline__ void load8(const float* p, float* x) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  }
  static __device__ __forceinline__ float load1(const float* p) { return *p; }
};

// ---------------------------------------------------------------------------
// Streaming loads through the global address space (global_load, not flat).
// Frag<T> holds one lane's 16 packed entries of one array in one chunk.
// ---------------------------------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 g_cu32x4;

template <bool LAST = false>
__device__ __forceinline__ uint4 gload16(const void* p) {
  // LAST: the data is not read again (non-temporal: no cache allocation)
  const u32x4 v = LAST ? __builtin_nontemporal_load((g_cu32x4*)(p)) : *(g_cu32x4*)(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <typename T>
struct Frag;
template <>
struct Frag<uint16_t> {
  uint4 q[2];
};
template <>
struct Frag<float> {
  uint4 q[4];
};

template <bool LAST, typename T>
__device__ __forceinline__ void frag_load(Frag<T>& f, const T* row, int c, int lane) {
  const T* p = row + c * CHUNK + 8 * lane;
  if constexpr (sizeof(T) == 2) {
    f.q[0] = gload16<LAST>(p);
    f.q[1] = gload16<LAST>(p + 512);
  } else {
    f.q[0] = gload16<LAST>(p);
    f.q[1] = gload16<LAST>(p + 4);
    f.q[2] = gload16<LAST>(p + 512);
    f.q[3] = gload16<LAST>(p + 516);
  }
}

__device__ __forceinline__ void unpack_bf16x8(const uint4 q, float* y) {
  y[0] = __uint_as_float(q.x << 16);
  y[1] = __uint_as_float(q.x & 0xffff0000u);
  y[2] = __uint_as_float(q.y << 16);
  y[3] = __uint_as_float(q.y & 0xffff0000u);
  y[4] = __uint_as_float(q.z << 16);
  y[5] = __uint_as_float(q.z & 0xffff0000u);
  y[6] = __uint_as_float(q.w << 16);
  y[7] = __uint_as_float(q.w & 0xffff0000u);
}

// x[e] in the elem_offset order.
__device__ __forceinline__ void frag_unpack(const Frag<uint16_t>& f, float* x) {
  unpack_bf16x8(f.q[0], x);
  unpack_bf16x8(f.q[1], x + 8);
}
__device__ __forceinline__ void frag_unpack(const Frag<float>& f, float* x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[4 * i + 0] = __uint_as_float(f.q[i].x);
    x[4 * i + 1] = __uint_as_float(f.q[i].y);
    x[4 * i + 2] = __uint_as_float(f.q[i].z);
    x[4 * i + 3] = __uint_as_float(f.q[i].w);
  }
}

// Loads the 16 entries of this lane in chunk c.  With TAIL the chunk may end
// before 1024 entries: missing entries are not read and their bit in *valid is 0.
template <typename T, bool TAIL>
__device__ __forceinline__ void load_lane(const T* row, int c, int lane, int V, float* x,
                                          uint32_t* valid) {
  const int base = c * CHUNK;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int v0 = base + h * 512 + 8 * lane;
    if (!TAIL || v0 + 8 <= V) {
      Loader<T>::load8(row + v0, x + 8 * h);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[8 * h + e] = (v0 + e < V) ? Loader<T>::load1(row + v0 + e) : 0.0f;
    }
  }
  if (TAIL) {
    uint32_t m = 0;
#pragma unroll
    for (int e = 0; e < EPL; ++e) m |= (base + elem_offset(lane, e) < V) ? (1u << e) : 0u;
    *valid = m;
  } else {
    *valid = 0xffffu;
  }
}

// ---------------------------------------------------------------------------
// Gradient stores (same lane layout as the loads).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;  // NaN
  const uint32_t rounding = 0x7fffu + ((u >> 16) & 1u);  // round to nearest even
  return (u + rounding) >> 16;
}

// Gradient rows are written once and not read back: non-temporal stores.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) f32x4 g_f32x4;
typedef __attribute__((address_space(1))) u32x4 g_u32x4;

template <typename G>
struct Storer;

template <>
struct Storer<float> {
  static __device__ __forceinline__ void store8(float* p, const float* x) {
    f32x4 a = {x[0], x[1], x[2], x[3]};
    f32x4 b = {x[4], x[5], x[6], x[7]};
    __builtin_nontemporal_store(a, (g_f32x4*)(p));
    __builtin_nontemporal_store(b, (g_f32x4*)(p + 4));
  }
  static __device__ __forceinline__ void store1(float* p, float x) { *p = x; }
};

template <>
struct Storer<uint16_t> {
  static __device__ __forceinline__ void store8(uint16_t* p, const float* x) {
    uint4 q;
    q.x = f32_to_bf16_bits(x[0]) | (f32_to_bf16_bits(x[1]) << 16);
    q.y = f32_to_bf16_bits(x[2]) | (f32_to_bf16_bits(x[3]) << 16);
    q.z = f32_to_bf16_bits(x[4]) | (f32_to_bf16_bits(x[5]) << 16);
    q.w = f32_to_bf16_bits(x[6]) | (f32_to_bf16_bits(x[7]) << 16);
    u32x4 v = {q.x, q.y, q.z, q.w};
    __builtin_nontemporal_store(v, (g_u32x4*)(p));
  }
  static __device__ __forceinline__ void store1(uint16_t* p, float x) {
    *p = static_cast<uint16_t>(f32_to_bf16_bits(x));
  }
};

template <typename G, bool TAIL>
__device__ __forceinline__ void store_lane(G* row, int c, int lane, int V, const float* x) {
  const int base = c * CHUNK;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int v0 = base + h * 512 + 8 * lane;
    if (!TAIL || v0 + 8 <= V) {
      Storer<G>::store8(row + v0, x + 8 * h);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (v0 + e < V) Storer<G>::store1(row + v0 + e, x[8 * h + e]);
    }
  }
}

// ---------------------------------------------------------------------------
// Wave reductions.  Inside each row of 16 lanes: DPP exchanges with the lane
// of index xor 1, xor 2, the half-row mirror and the row mirror (after which
// the row is uniform); then the four row values, read as scalars, are
// combined in a fixed order.  Every lane ends with the same bits.
// ---------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const int lo = __builtin_amdgcn_mov_dpp(static_cast<int>(static_cast<uint32_t>(u)), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(static_cast<int>(static_cast<uint32_t>(u >> 32)), CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(double, (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
__device__ __forceinline__ double lane_d(double v, int l) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(u)), l));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(u >> 32)), l));
  return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
}

constexpr int DPP_XOR1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <-> 7 - i in each half row
constexpr int DPP_MIRROR = 0x140;      // lane i <-> 15 - i in each row

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<DPP_XOR1>(v));
  v = fmaxf(v, dpp_f<DPP_XOR2>(v));
  v = fmaxf(v, dpp_f<DPP_HALF_MIRROR>(v));
  v = fmaxf(v, dpp_f<DPP_MIRROR>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<DPP_XOR1>(v);
  v += dpp_f<DPP_XOR2>(v);
  v += dpp_f<DPP_HALF_MIRROR>(v);
  v += dpp_f<DPP_MIRROR>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
__device__ __forceinline__ double wave_sum(double v) {
  v += dpp_d<DPP_XOR1>(v);
  v += dpp_d<DPP_XOR2>(v);
  v += dpp_d<DPP_HALF_MIRROR>(v);
  v += dpp_d<DPP_MIRROR>(v);
  return (lane_d(v, 0) + lane_d(v, 16)) + (lane_d(v, 32) + lane_d(v, 48));
}
__device__ __forceinline__ int wave_min(int v) {
  v = min(v, dpp_i<DPP_XOR1>(v));
  v = min(v, dpp_i<DPP_XOR2>(v));
  v = min(v, dpp_i<DPP_HALF_MIRROR>(v));
  v = min(v, dpp_i<DPP_MIRROR>(v));
  return min(min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16)),
             min(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48)));
}
// true on every lane if pred holds on any active lane
__device__ __forceinline__ bool wave_any(bool pred) { return __ballot(pred) != 0; }
// (key, index) minimum; ties go to the lower index.
__device__ __forceinline__ void wave_argmin(float& key, int& idx) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    const float k2 = __shfl_xor(key, o, WAVE);
    const int i2 = __shfl_xor(idx, o, WAVE);
    if (k2 < key || (k2 == key && i2 < idx)) { key = k2; idx = i2; }
  }
}
__device__ __forceinline__ void wave_argmin(double& key, int& idx) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    const double k2 = __shfl_xor(key, o, WAVE);
    const int i2 = __shfl_xor(idx, o, WAVE);
    if (k2 < key || (k2 == key && i2 < idx)) { key = k2; idx = i2; }
  }
}
// (value, index) maximum; ties go to the lower index.
__device__ __forceinline__ void wave_argmax(float& val, int& idx) {
#pragma unroll
  for (int o = WAVE / 2; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(val, o, WAVE);
    const int i2 = __shfl_xor(idx, o, WAVE);
    if (v2 > val || (v2 == val && i2 < idx)) { val = v2; idx = i2; }
  }
}

// ---------------------------------------------------------------------------
// Philox-4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) and the stream layout:
// key = (seed lo, seed hi), counter = (block j, stream, g lo, g hi); the four
// words of block j are the uniforms for indices 4j .. 4j+3 of the stream.
// ---------------------------------------------------------------------------
enum Stream : uint32_t {
  PROP_CHUNK = 0, PROP_ELEM = 1, ACCEPT = 2, RES_CHUNK = 3, RES_ELEM = 4,
  TS_CHUNK = 5, TS_ELEM = 6,  // teacher-sampled correction target
  SELECT = 7                  // placement controls, index 0 of each position
};

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z);
    const uint32_t lo1 = 0xCD9E8D57u * c.z;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// u = (2*(x >> 9) + 1) * 2^-24, in (0, 1), exact in float.
__device__ __forceinline__ float word_to_uniform(uint32_t x) {
  return static_cast<float>(2u * (x >> 9) + 1u) * 0x1p-24f;
}

// Block j of (seed, stream, g): the words of indices 4j .. 4j+3.
__device__ __forceinline__ uint4 philox_block(uint64_t seed, uint32_t stream, uint64_t g, uint32_t j) {
  return philox4x32_10(make_uint4(j, stream, static_cast<uint32_t>(g), static_cast<uint32_t>(g >> 32)),
                       static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
}

__device__ __forceinline__ float philox_uniform(uint64_t seed, uint32_t stream, uint64_t g,
                                                uint32_t index) {
  const uint4 w = philox_block(seed, stream, g, index >> 2);
  const uint32_t sel = index & 3u;
  const uint32_t x = sel == 0 ? w.x : sel == 1 ? w.y : sel == 2 ? w.z : w.w;
  return word_to_uniform(x);
}

}  // namespace saki
