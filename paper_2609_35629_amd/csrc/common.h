// Device helpers shared by the santapp kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace santapp {

constexpr int kWave = 64;

// Element types of K/V rows.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Low / high bf16 of a packed 32-bit word, widened exactly to fp32.
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// 16-byte streaming loads: K/V rows are read once per decode step, so they
// are fetched without displacing the rest of the cache contents.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const void* p) {
    const u32x4_t v = __builtin_nontemporal_load(static_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float4 load_stream_f(const void* p) {
    const f32x4_t v = __builtin_nontemporal_load(static_cast<const f32x4_t*>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint2 load_stream8(const void* p) {
    typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
    const u32x2_t v = __builtin_nontemporal_load(static_cast<const u32x2_t*>(p));
    return make_uint2(v.x, v.y);
}

// Streaming stores of values written once and read once by the next kernel.
__device__ __forceinline__ void store_stream(float* p, float4 v) {
    __builtin_nontemporal_store(f32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<f32x4_t*>(p));
}

__device__ __forceinline__ void store_stream2(float* p, float2 v) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    __builtin_nontemporal_store(f32x2_t{v.x, v.y}, reinterpret_cast<f32x2_t*>(p));
}

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, size_t i);

template <>
__device__ __forceinline__ float load_elem<bf16_t>(const bf16_t* p, size_t i) {
    return bf16_to_f32(p[i].bits);
}

template <>
__device__ __forceinline__ float load_elem<float>(const float* p, size_t i) {
    return p[i];
}

// A lane's DPL consecutive elements of a routing-key row (16 lanes per
// row), widened to fp32 exactly.
template <typename T, int DPL>
struct RepChunk;

template <>
struct RepChunk<bf16_t, 8> {
    using raw = uint4;
    static __device__ __forceinline__ raw load(const bf16_t* p) { return load_stream(p); }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const uint32_t w = (e < 2) ? r.x : (e < 4) ? r.y : (e < 6) ? r.z : r.w;
        return (e & 1) ? bf16hi(w) : bf16lo(w);
    }
};

template <>
struct RepChunk<bf16_t, 4> {
    using raw = uint2;
    static __device__ __forceinline__ raw load(const bf16_t* p) { return load_stream8(p); }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const uint32_t w = (e < 2) ? r.x : r.y;
        return (e & 1) ? bf16hi(w) : bf16lo(w);
    }
};

template <>
struct RepChunk<float, 8> {
    struct raw {
        float4 a, b;
    };
    static __device__ __forceinline__ raw load(const float* p) {
        raw r;
        r.a = load_stream_f(p);
        r.b = load_stream_f(p + 4);
        return r;
    }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        const float4& v = (e < 4) ? r.a : r.b;
        const int k = e & 3;
        return k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
    }
};

template <>
struct RepChunk<float, 4> {
    using raw = float4;
    static __device__ __forceinline__ raw load(const float* p) { return load_stream_f(p); }
    static __device__ __forceinline__ float get(const raw& r, int e) {
        return e == 0 ? r.x : e == 1 ? r.y : e == 2 ? r.z : r.w;
    }
};

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11).  One round maps
// (x0,x1,x2,x3) to (hi(M1 x2)^x1^k0, lo(M1 x2), hi(M0 x0)^x3^k1, lo(M0 x0));
// the key advances by the Weyl increments between rounds.
// ---------------------------------------------------------------------------
struct u64x4 {
    uint64_t v[4];
};

// The 128-bit product of two 64-bit words from four independent 32 x 32-bit
// partial products (each one multiply-add on the vector ALU).
__device__ __forceinline__ void mul64_wide(uint64_t a, uint64_t b, uint64_t& lo, uint64_t& hi) {
    const uint64_t a0 = a & 0xffffffffull, a1 = a >> 32, b0 = b & 0xffffffffull, b1 = b >> 32;
    const uint64_t p00 = a0 * b0, p01 = a0 * b1, p10 = a1 * b0, p11 = a1 * b1;
    const uint64_t mid = (p00 >> 32) + (p01 & 0xffffffffull) + (p10 & 0xffffffffull);
    lo = (mid << 32) | (p00 & 0xffffffffull);
    hi = p11 + (p01 >> 32) + (p10 >> 32) + (mid >> 32);
}

__device__ __forceinline__ u64x4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                               uint64_t k0, uint64_t k1) {
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
    // kept rolled: the round is a handful of 64-bit multiplies and the loop
    // overhead is one scalar add and branch, so unrolling buys little code
    // speed for ten times the code size
#pragma unroll 1
    for (int r = 0; r < 10; ++r) {
        if (r) {
            k0 += W0;
            k1 += W1;
        }
        uint64_t lo0, hi0, lo1, hi1;
        mul64_wide(M0, c0, lo0, hi0);
        mul64_wide(M1, c2, lo1, hi1);
        const uint64_t n0 = hi1 ^ c1 ^ k0;
        const uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
    }
    u64x4 o;
    o.v[0] = c0;
    o.v[1] = c1;
    o.v[2] = c2;
    o.v[3] = c3;
    return o;
}

// Standard Gumbel variate of a 64-bit Philox word w: U = ((w >> 12) + 1/2)
// 2^-52 is exact and inside (0, 1); G = -log(-log U).
__device__ __forceinline__ double gumbel_of_word(uint64_t w) {
    const double u = (static_cast<double>(w >> 12) + 0.5) * 0x1.0p-52;
    return -log(-log(u));
}

// The variate of team g for (seed, step, b, h) is that of word g % 4 of the
// block at counter (g / 4, h, b, step), key (seed, 0); one block serves
// teams 4 (g / 4) .. 4 (g / 4) + 3.

// Order-preserving map of a double onto uint64 (larger value -> larger key).
__device__ __forceinline__ uint64_t order_key(double y) {
    const uint64_t b = static_cast<uint64_t>(__double_as_longlong(y));
    return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ double key_value(uint64_t k) {
    const uint64_t b = (k >> 63) ? (k & 0x7fffffffffffffffull) : ~k;
    return __longlong_as_double(static_cast<long long>(b));
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    const int lane = threadIdx.x & (kWave - 1);
    return (lane == 0) ? 0ull : (~0ull >> (64 - lane));
}

__device__ __forceinline__ int wave_id() { return threadIdx.x / kWave; }
__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// DPP row rotations (within each 16-lane row of the wave): row_ror:n is
// control word 0x120 + n.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(b & 0xffffffff), CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(b >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((static_cast<long long>(hi) << 32) |
                                static_cast<long long>(static_cast<unsigned>(lo)));
}

// Sum over the 16 lanes of a DPP row; every lane of the row receives it.
__device__ __forceinline__ float row16_sum(float v) {
    v += dpp_f32<0x128>(v);
    v += dpp_f32<0x124>(v);
    v += dpp_f32<0x122>(v);
    v += dpp_f32<0x121>(v);
    return v;
}

// Inclusive prefix sum over the 64 lanes of the wave (row shifts inside each
// 16-lane row, then row broadcasts of lane 15 and lane 31).
__device__ __forceinline__ int wave_incl_scan(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);  // row_shr:1
    x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);  // row_shr:2
    x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);  // row_shr:4
    x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);  // row_shr:8
    x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15
    x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return x;
}

__device__ __forceinline__ int readlane(int x, int lane) { return __builtin_amdgcn_readlane(x, lane); }

__device__ __forceinline__ uint64_t readlane(uint64_t x, int lane) {
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(x & 0xffffffffu), lane);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(x >> 32), lane);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Sum over all 64 lanes; the result is wave-uniform.
__device__ __forceinline__ int wave_sum(int x) {
    x += __builtin_amdgcn_update_dpp(0, x, 0x128, 0xF, 0xF, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x124, 0xF, 0xF, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x122, 0xF, 0xF, false);
    x += __builtin_amdgcn_update_dpp(0, x, 0x121, 0xF, 0xF, false);
    return readlane(x, 0) + readlane(x, 16) + readlane(x, 32) + readlane(x, 48);
}

template <bool kAnd>
__device__ __forceinline__ uint32_t wave_bits32(uint32_t x) {
    int v = static_cast<int>(x);
#define SANTAPP_BITSTEP(CTRL)                                                            \
    {                                                                                    \
        const int t = __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);         \
        v = kAnd ? (v & t) : (v | t);                                                    \
    }
    SANTAPP_BITSTEP(0x128)
    SANTAPP_BITSTEP(0x124)
    SANTAPP_BITSTEP(0x122)
    SANTAPP_BITSTEP(0x121)
#undef SANTAPP_BITSTEP
    const uint32_t a = readlane(v, 0), b = readlane(v, 16), c = readlane(v, 32), d = readlane(v, 48);
    return kAnd ? (a & b & c & d) : (a | b | c | d);
}

// Bitwise AND / OR of a 64-bit value over all 64 lanes (wave-uniform).
__device__ __forceinline__ uint64_t wave_and64(uint64_t x) {
    return (static_cast<uint64_t>(wave_bits32<true>(static_cast<uint32_t>(x >> 32))) << 32) |
           wave_bits32<true>(static_cast<uint32_t>(x));
}

__device__ __forceinline__ uint64_t wave_or64(uint64_t x) {
    return (static_cast<uint64_t>(wave_bits32<false>(static_cast<uint32_t>(x >> 32))) << 32) |
           wave_bits32<false>(static_cast<uint32_t>(x));
}

template <bool kMin>
__device__ __forceinline__ uint64_t wave_ext64(uint64_t x) {
#define SANTAPP_EXTSTEP(CTRL)                                                                    \
    {                                                                                            \
        const uint32_t lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(x & 0xffffffffu), CTRL, \
                                                        0xF, 0xF, false);                         \
        const uint32_t hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(x >> 32), CTRL, 0xF,  \
                                                        0xF, false);                              \
        const uint64_t y = (static_cast<uint64_t>(hi) << 32) | lo;                               \
        x = kMin ? (y < x ? y : x) : (y > x ? y : x);                                            \
    }
    SANTAPP_EXTSTEP(0x128)
    SANTAPP_EXTSTEP(0x124)
    SANTAPP_EXTSTEP(0x122)
    SANTAPP_EXTSTEP(0x121)
#undef SANTAPP_EXTSTEP
    uint64_t r = readlane(x, 0);
#pragma unroll
    for (int row = 1; row < 4; ++row) {
        const uint64_t y = readlane(x, 16 * row);
        r = kMin ? (y < r ? y : r) : (y > r ? y : r);
    }
    return r;
}

// Unsigned 64-bit minimum / maximum over all 64 lanes (wave-uniform).
__device__ __forceinline__ uint64_t wave_min64(uint64_t x) { return wave_ext64<true>(x); }
__device__ __forceinline__ uint64_t wave_max64(uint64_t x) { return wave_ext64<false>(x); }

__device__ __forceinline__ double row16_sum(double v) {
    v += dpp_f64<0x128>(v);
    v += dpp_f64<0x124>(v);
    v += dpp_f64<0x122>(v);
    v += dpp_f64<0x121>(v);
    return v;
}

}  // namespace santapp
