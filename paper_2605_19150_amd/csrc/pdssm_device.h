// pdssm_device.h -- wave-level building blocks of the PD scan for gfx950.
//
// One 64-lane wavefront owns one sequence's N-wide complex state.  State
// entry j lives in lane j / SL, slot j % SL, where SL = max(1, N/64) entries
// per lane (consecutive entries per lane so a step's row of D, b or c is one
// 8*SL-byte vector load per lane).  For N < 64 only the first N lanes are
// active.  Cross-lane movement goes through a per-wave LDS buffer; LDS
// instructions of one wave execute in issue order, so a wave needs no
// workgroup barrier for its own buffer, only a compiler fence (wave_sync).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pdssm_io.h"

namespace pdssm {

constexpr int kWave = 64;
constexpr int kErrIndex = -5;  // PDSSM_ERR_INDEX

template <int N>
struct Lay {
    static constexpr int SL = N > kWave ? N / kWave : 1;     // entries per lane
    static constexpr int LANES = N < kWave ? N : kWave;      // active lanes
    static_assert(N >= 8 && N <= 256 && (N & (N - 1)) == 0, "N must be a power of two in [8,256]");
};

// ------------------------------------------------------------------ complex
// Complex products with explicit fused multiply-adds: the rounding is fixed
// by the source, not by where the compiler chooses to contract, so every
// kernel variant (e.g. fp32 or bf16 input/output) computes the same bits.
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
    return make_float2(fmaf(a.x, b.x, -(a.y * b.y)), fmaf(a.x, b.y, a.y * b.x));
}
// conj(a) * b
__device__ __forceinline__ float2 cmulc(float2 a, float2 b) {
    return make_float2(fmaf(a.x, b.x, a.y * b.y), fmaf(a.x, b.y, -(a.y * b.x)));
}
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }

// The same operations on the real-valued model's float elements.  Each
// rounds as the complex one does on values whose imaginary parts are 0 (a
// complex product's real part is then fmaf(a, b, -0), the rounded product),
// and every product that feeds a sum goes through one of the explicit
// multiply-adds below in both forms, so the two element types compute the
// same bits on real data.
__device__ __forceinline__ float cmul(float a, float b) { return a * b; }
__device__ __forceinline__ float cmulc(float a, float b) { return a * b; }
__device__ __forceinline__ float cadd(float a, float b) { return a + b; }

// acc + a b and acc + conj(a) b, real and imaginary parts each as two
// chained fused multiply-adds (for real data the second adds an exact 0).
__device__ __forceinline__ float2 cfma(float2 acc, float2 a, float2 b) {
    return make_float2(fmaf(-a.y, b.y, fmaf(a.x, b.x, acc.x)), fmaf(a.y, b.x, fmaf(a.x, b.y, acc.y)));
}
__device__ __forceinline__ float2 cfmac(float2 acc, float2 a, float2 b) {
    return make_float2(fmaf(a.y, b.y, fmaf(a.x, b.x, acc.x)), fmaf(-a.y, b.x, fmaf(a.x, b.y, acc.y)));
}
__device__ __forceinline__ float cfma(float acc, float a, float b) { return fmaf(a, b, acc); }
__device__ __forceinline__ float cfmac(float acc, float a, float b) { return fmaf(a, b, acc); }

// acc + Re(c h): the readout term c.x h.x - c.y h.y.
__device__ __forceinline__ float re_fma(float acc, float2 c, float2 h) { return fmaf(-c.y, h.y, fmaf(c.x, h.x, acc)); }
__device__ __forceinline__ float re_fma(float acc, float c, float h) { return fmaf(c, h, acc); }

// Element constants.
template <class E>
__device__ __forceinline__ E ezero() {
    if constexpr (sizeof(E) == 8) return make_float2(0.f, 0.f);
    else return 0.f;
}
template <class E>
__device__ __forceinline__ E eone() {
    if constexpr (sizeof(E) == 8) return make_float2(1.f, 0.f);
    else return 1.f;
}
// g + s conj(c) (the backward's readout term dy_t conj(c_t))
__device__ __forceinline__ float2 add_sconj(float2 g, float s, float2 c) {
    return make_float2(fmaf(s, c.x, g.x), fmaf(-s, c.y, g.y));
}
__device__ __forceinline__ float add_sconj(float g, float s, float c) { return fmaf(s, c, g); }
// s conj(h) (the readout gradient dc_t = dy_t conj(h_t))
__device__ __forceinline__ float2 sconj(float s, float2 h) { return make_float2(s * h.x, -s * h.y); }
__device__ __forceinline__ float sconj(float s, float h) { return s * h; }

// ------------------------------------------------------------------ wave sync
// Orders this wave's LDS accesses in the compiler; the hardware already
// executes one wave's LDS instructions in order.
__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Index of this wave in its workgroup, as a wave-uniform (scalar) value: the
// compiler cannot prove threadIdx.x >> 6 uniform, and everything derived from
// it (chunk numbers, row addresses, loop bounds) would otherwise live in
// vector registers and branch per lane.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

__device__ __forceinline__ int readlane_i(int v, int l) { return __builtin_amdgcn_readlane(v, l); }
__device__ __forceinline__ float readlane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ float readlane_e(float v, int l) { return readlane_f(v, l); }
__device__ __forceinline__ float2 readlane_e(float2 v, int l) {
    return make_float2(readlane_f(v.x, l), readlane_f(v.y, l));
}

// Sum over the 64 lanes; the total lands in lane 63 (other lanes hold
// partial sums).  Row-wise inclusive scan with DPP row_shr, then the
// row_bcast15 / row_bcast31 steps carry row totals up to the last row.
__device__ __forceinline__ float wave_sum_last(float v) {
    float t;
    t = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x111, 0xf, 0xf, true));
    v += t;
    t = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x112, 0xf, 0xf, true));
    v += t;
    t = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x114, 0xf, 0xf, true));
    v += t;
    t = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x118, 0xf, 0xf, true));
    v += t;
    t = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x142, 0xa, 0xf, false));
    v += t;
    t = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x143, 0xc, 0xf, false));
    v += t;
    return v;
}

// Forces a value to be computed before this point: the compiler otherwise
// sinks work to its first use, which may sit behind a wait on another wave.
__device__ __forceinline__ void materialize(float v) { asm volatile("" ::"v"(v) : "memory"); }
__device__ __forceinline__ void materialize(int v) { asm volatile("" ::"v"(v) : "memory"); }
__device__ __forceinline__ void materialize(float2 v) {
    materialize(v.x);
    materialize(v.y);
}

// Keeps memory operations issued before this point from being moved below it
// (e.g. a prefetch the compiler would otherwise sink to its first use).
__device__ __forceinline__ void issue_fence() { asm volatile("" ::: "memory"); }

// ------------------------------------------------------------------ per-lane vectors
template <int SL, class E = float2>
struct CV {
    E v[SL];
};
template <int SL>
struct IV {
    int v[SL];
};

template <int SL, class E = float2>
__device__ __forceinline__ CV<SL, E> cv_zero() {
    CV<SL, E> r;
#pragma unroll
    for (int s = 0; s < SL; ++s) r.v[s] = ezero<E>();
    return r;
}

// This lane's SL consecutive float entries of a row (row + lane*SL), as one
// vector access.
template <int SL>
__device__ __forceinline__ CV<SL, float> ld_cv(const float* __restrict__ row, int lane) {
    CV<SL, float> r;
    const float* p = row + lane * SL;
    if constexpr (SL == 1) {
        r.v[0] = *p;
    } else if constexpr (SL == 2) {
        const float2 q = *reinterpret_cast<const float2*>(p);
        r.v[0] = q.x;
        r.v[1] = q.y;
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4) {
            const float4 q = *reinterpret_cast<const float4*>(p + s);
            r.v[s] = q.x;
            r.v[s + 1] = q.y;
            r.v[s + 2] = q.z;
            r.v[s + 3] = q.w;
        }
    }
    return r;
}
template <int SL>
__device__ __forceinline__ void st_cv(float* __restrict__ row, int lane, const CV<SL, float>& x) {
    float* p = row + lane * SL;
    if constexpr (SL == 1) {
        *p = x.v[0];
    } else if constexpr (SL == 2) {
        *reinterpret_cast<float2*>(p) = make_float2(x.v[0], x.v[1]);
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4)
            *reinterpret_cast<float4*>(p + s) = make_float4(x.v[s], x.v[s + 1], x.v[s + 2], x.v[s + 3]);
    }
}

// Load this lane's SL consecutive complex entries of a row (row + lane*SL).
template <int SL>
__device__ __forceinline__ CV<SL> ld_cv(const float2* __restrict__ row, int lane) {
    CV<SL> r;
    const float2* p = row + lane * SL;
    if constexpr (SL == 1) {
        r.v[0] = *p;
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 2) {
            float4 q = *reinterpret_cast<const float4*>(p + s);
            r.v[s] = make_float2(q.x, q.y);
            r.v[s + 1] = make_float2(q.z, q.w);
        }
    }
    return r;
}

// Raw buffer access to rows of a [.., N] complex tensor: a scalar resource
// descriptor holds the base of a block of rows, a scalar offset selects the
// row and one shared 32-bit VGPR holds the lane's byte offset, so a chunk of
// row loads costs no per-load 64-bit address registers.  Callers keep every
// row inside the tensor; a load through a zero-size descriptor returns 0.
constexpr int kBufferDword3 = 0x00020000;  // raw buffer, gfx9 family
// Cache-policy operand of a load that streams data read exactly once: the
// nontemporal hint (nt) of gfx94x/gfx950.
constexpr int kLoadStream = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_block(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kBufferDword3);
}

// This lane's SL consecutive complex entries of the row at byte offset soff;
// AUX is the cache-policy operand (0 or kLoadStream).
template <int SL, int AUX = 0>
__device__ __forceinline__ CV<SL> ld_row(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    CV<SL> out;
    if constexpr (SL == 1) {
        out.v[0] = __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX));
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 2) {
            const float4 q =
                __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff + 8 * s, AUX));
            out.v[s] = make_float2(q.x, q.y);
            out.v[s + 1] = make_float2(q.z, q.w);
        }
    }
    return out;
}

// Complex64 rows in memory (states: h0, saved, h_final, dh0, segment
// aggregates) as elements: the real model keeps the real part and writes
// imaginary parts 0.
template <class E, int SL>
__device__ __forceinline__ CV<SL, E> to_elem(const CV<SL>& x) {
    if constexpr (sizeof(E) == 8) {
        return x;
    } else {
        CV<SL, E> r;
#pragma unroll
        for (int s = 0; s < SL; ++s) r.v[s] = x.v[s].x;
        return r;
    }
}
template <int SL, class E>
__device__ __forceinline__ CV<SL> to_c64(const CV<SL, E>& x) {
    if constexpr (sizeof(E) == 8) {
        return x;
    } else {
        CV<SL> r;
#pragma unroll
        for (int s = 0; s < SL; ++s) r.v[s] = make_float2(x.v[s], 0.f);
        return r;
    }
}
template <class E, int SL>
__device__ __forceinline__ CV<SL, E> ld_state(const float2* __restrict__ row, int lane) {
    return to_elem<E>(ld_cv<SL>(row, lane));
}
template <int SL, class E>
__device__ __forceinline__ void st_state(float2* __restrict__ row, int lane, const CV<SL, E>& x) {
    st_cv<SL>(row, lane, to_c64<SL>(x));
}

// Chunk-entering states (the saved states, their LDS staging and the
// multi-pass carries): complex64 rows, or float32 rows for the real model,
// whose states are real.  off counts entries from base.
template <int SL, class E>
__device__ __forceinline__ CV<SL, E> ld_srow(const float2* base, size_t off, int lane) {
    if constexpr (sizeof(E) == sizeof(float)) return ld_cv<SL>(reinterpret_cast<const float*>(base) + off, lane);
    else return ld_cv<SL>(base + off, lane);
}
template <int SL, class E>
__device__ __forceinline__ void st_srow(float2* base, size_t off, int lane, const CV<SL, E>& x) {
    if constexpr (sizeof(E) == sizeof(float)) st_cv<SL>(reinterpret_cast<float*>(base) + off, lane, x);
    else st_cv<SL>(base + off, lane, x);
}

// ------------------------------------------------------------------ bf16 (re, im) pairs
// A complex value in 32 bits: bf16 real part in the low half, bf16 imaginary
// part in the high half (torch: view_as_real(x).to(bfloat16)).  Widening is
// exact; narrowing rounds each part to nearest, ties to even (finite values).
__device__ __forceinline__ float2 bf2_to_f2(uint32_t w) {
    return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xffff0000u));
}
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float v) {
    const uint32_t u = __float_as_uint(v);
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t f2_to_bf2(float2 v) {
    return f32_to_bf16_bits(v.x) | (f32_to_bf16_bits(v.y) << 16);
}

// One 4-byte entry widened to a complex value, and back (the real format
// keeps the real part only).
template <int IO>
__device__ __forceinline__ float2 word_to_f2(uint32_t w) {
    static_assert(IO == kIoBf16 || IO == kIoReal, "4-byte formats only");
    if constexpr (IO == kIoBf16) return bf2_to_f2(w);
    else return make_float2(__uint_as_float(w), 0.f);
}
template <int IO>
__device__ __forceinline__ uint32_t f2_to_word(float2 v) {
    static_assert(IO == kIoBf16 || IO == kIoReal, "4-byte formats only");
    if constexpr (IO == kIoBf16) return f2_to_bf2(v);
    else return __float_as_uint(v.x);
}

// ld_row for rows of 4-byte entries (bf16 pairs or real fp32).
template <int SL, int AUX, int IO>
__device__ __forceinline__ CV<SL> ld_row_w(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    CV<SL> out;
    if constexpr (SL == 1) {
        out.v[0] = word_to_f2<IO>(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX));
    } else if constexpr (SL == 2) {
        const uint2 q = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX));
        out.v[0] = word_to_f2<IO>(q.x);
        out.v[1] = word_to_f2<IO>(q.y);
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4) {
            const uint4 q =
                __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff + 4 * s, AUX));
            out.v[s] = word_to_f2<IO>(q.x);
            out.v[s + 1] = word_to_f2<IO>(q.y);
            out.v[s + 2] = word_to_f2<IO>(q.z);
            out.v[s + 3] = word_to_f2<IO>(q.w);
        }
    }
    return out;
}

// The real-valued model's rows as float elements (no widening).
template <int SL, int AUX>
__device__ __forceinline__ CV<SL, float> ld_row_r(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    CV<SL, float> out;
    if constexpr (SL == 1) {
        out.v[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX));
    } else if constexpr (SL == 2) {
        const uint2 q = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX));
        out.v[0] = __uint_as_float(q.x);
        out.v[1] = __uint_as_float(q.y);
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4) {
            const uint4 q =
                __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff + 4 * s, AUX));
            out.v[s] = __uint_as_float(q.x);
            out.v[s + 1] = __uint_as_float(q.y);
            out.v[s + 2] = __uint_as_float(q.z);
            out.v[s + 3] = __uint_as_float(q.w);
        }
    }
    return out;
}

// A row of float elements written with the nontemporal hint (the real
// model's gradient rows).
template <int SL>
__device__ __forceinline__ void st_row_r_stream(float* __restrict__ row, int lane, const CV<SL, float>& x) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    float* p = row + lane * SL;
    if constexpr (SL == 1) {
        __builtin_nontemporal_store(x.v[0], p);
    } else if constexpr (SL == 2) {
        __builtin_nontemporal_store(f32x2{x.v[0], x.v[1]}, reinterpret_cast<f32x2*>(p));
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4)
            __builtin_nontemporal_store(f32x4{x.v[s], x.v[s + 1], x.v[s + 2], x.v[s + 3]},
                                        reinterpret_cast<f32x4*>(p + s));
    }
}

// This lane's SL entries of a row of 4-byte entries (row + lane*SL), with the
// nontemporal hint (rows written once).
template <int SL, int IO>
__device__ __forceinline__ void st_row_w_stream(uint32_t* __restrict__ row, int lane, const CV<SL>& x) {
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    uint32_t* p = row + lane * SL;
    if constexpr (SL == 1) {
        __builtin_nontemporal_store(f2_to_word<IO>(x.v[0]), p);
    } else if constexpr (SL == 2) {
        __builtin_nontemporal_store(u32x2{f2_to_word<IO>(x.v[0]), f2_to_word<IO>(x.v[1])},
                                    reinterpret_cast<u32x2*>(p));
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4)
            __builtin_nontemporal_store(u32x4{f2_to_word<IO>(x.v[s]), f2_to_word<IO>(x.v[s + 1]),
                                              f2_to_word<IO>(x.v[s + 2]), f2_to_word<IO>(x.v[s + 3])},
                                        reinterpret_cast<u32x4*>(p + s));
    }
}

template <int SL>
__device__ __forceinline__ void st_cv(float2* __restrict__ row, int lane, const CV<SL>& x) {
    float2* p = row + lane * SL;
    if constexpr (SL == 1) {
        *p = x.v[0];
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 2)
            *reinterpret_cast<float4*>(p + s) = make_float4(x.v[s].x, x.v[s].y, x.v[s + 1].x, x.v[s + 1].y);
    }
}

// st_cv with the nontemporal hint, for output rows written once and never
// read back by the kernel.  Global stores, not raw buffer stores: a buffer
// store of more than 8 bytes with a scalar-register offset has shown its data
// registers overwritten before the store read them on gfx950 (the compiler
// inserts no wait state for that form).
template <int SL>
__device__ __forceinline__ void st_cv_stream(float2* __restrict__ row, int lane, const CV<SL>& x) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    float2* p = row + lane * SL;
    if constexpr (SL == 1) {
        __builtin_nontemporal_store(f32x2{x.v[0].x, x.v[0].y}, reinterpret_cast<f32x2*>(p));
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 2)
            __builtin_nontemporal_store(f32x4{x.v[s].x, x.v[s].y, x.v[s + 1].x, x.v[s + 1].y},
                                        reinterpret_cast<f32x4*>(p + s));
    }
}

template <int SL>
__device__ __forceinline__ IV<SL> ld_iv(const int* __restrict__ row, int lane) {
    IV<SL> r;
    const int* p = row + lane * SL;
    if constexpr (SL == 1) {
        r.v[0] = *p;
    } else if constexpr (SL == 2) {
        int2 q = *reinterpret_cast<const int2*>(p);
        r.v[0] = q.x;
        r.v[1] = q.y;
    } else {
#pragma unroll
        for (int s = 0; s < SL; s += 4) {
            int4 q = *reinterpret_cast<const int4*>(p + s);
            r.v[s] = q.x;
            r.v[s + 1] = q.y;
            r.v[s + 2] = q.z;
            r.v[s + 3] = q.w;
        }
    }
    return r;
}

template <int SL>
__device__ __forceinline__ void st_iv(int* __restrict__ row, int lane, const IV<SL>& x) {
#pragma unroll
    for (int s = 0; s < SL; ++s) row[lane * SL + s] = x.v[s];
}

// Replace out-of-range map entries by 0; returns true if any entry was bad.
template <int N, int SL>
__device__ __forceinline__ bool sanitize_map(IV<SL>& p) {
    bool bad = false;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        bool b = (unsigned)p.v[s] >= (unsigned)N;
        bad |= b;
        p.v[s] = b ? 0 : p.v[s];
    }
    return bad;
}

__device__ __forceinline__ void report_index_error(int* status) {
    if (status) *status = kErrIndex;
}

// ------------------------------------------------------------------ lane scans
// DPP move with zero for lanes outside the row mask or without a source.
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, ROWS, 0xf, true);
}
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_fr(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROWS, 0xf, true));
}

// Inclusive prefix sum of an int over the 64 lanes.
__device__ __forceinline__ int wave_incl_scan_i(int v) {
    v += dpp_i<0x111, 0xf>(v);
    v += dpp_i<0x112, 0xf>(v);
    v += dpp_i<0x114, 0xf>(v);
    v += dpp_i<0x118, 0xf>(v);
    v += dpp_i<0x142, 0xa>(v);
    v += dpp_i<0x143, 0xc>(v);
    return v;
}

// One step of the segmented scan: add the value DPP brings in when `take`.
template <int CTRL, int ROWS>
__device__ __forceinline__ void seg_step(float2& v, bool take) {
    const float tx = dpp_fr<CTRL, ROWS>(v.x), ty = dpp_fr<CTRL, ROWS>(v.y);
    v.x += take ? tx : 0.f;
    v.y += take ? ty : 0.f;
}

__device__ __forceinline__ void seg_step1(float& v, float t, bool take) { v += take ? t : 0.f; }

// Inclusive segmented sum over the 64 lanes of a complex value: a lane whose
// bit is set in `starts` begins a new segment (lane 0 always does).  Row-wise
// shifts, then the row broadcasts carry row totals across rows, each term
// taken only when its source lane lies in the same segment.
__device__ __forceinline__ float2 wave_seg_scan(float2 v, uint64_t starts, int lane) {
    const uint64_t le = starts & ((2ull << lane) - 1ull);  // lane 63: 2 << 63 wraps to 0
    const int s0 = le ? 63 - __builtin_clzll(le) : 0;      // first lane of this lane's segment
    seg_step<0x111, 0xf>(v, lane - 1 >= s0);
    seg_step<0x112, 0xf>(v, lane - 2 >= s0);
    seg_step<0x114, 0xf>(v, lane - 4 >= s0);
    seg_step<0x118, 0xf>(v, lane - 8 >= s0);
    seg_step<0x142, 0xa>(v, s0 < (lane & ~15));
    seg_step<0x143, 0xc>(v, s0 < 32);
    return v;
}

// The same for a real value (the real model's elements).
__device__ __forceinline__ float wave_seg_scan(float v, uint64_t starts, int lane) {
    const uint64_t le = starts & ((2ull << lane) - 1ull);
    const int s0 = le ? 63 - __builtin_clzll(le) : 0;
    seg_step1(v, dpp_fr<0x111, 0xf>(v), lane - 1 >= s0);
    seg_step1(v, dpp_fr<0x112, 0xf>(v), lane - 2 >= s0);
    seg_step1(v, dpp_fr<0x114, 0xf>(v), lane - 4 >= s0);
    seg_step1(v, dpp_fr<0x118, 0xf>(v), lane - 8 >= s0);
    seg_step1(v, dpp_fr<0x142, 0xa>(v), s0 < (lane & ~15));
    seg_step1(v, dpp_fr<0x143, 0xc>(v), s0 < 32);
    return v;
}
__device__ __forceinline__ float2 lane_up(float2 C) {  // from lane - 1
    return make_float2(dpp_fr<0x138, 0xf>(C.x), dpp_fr<0x138, 0xf>(C.y));
}
__device__ __forceinline__ float lane_up(float C) { return dpp_fr<0x138, 0xf>(C); }

// ------------------------------------------------------------------ collisions in a fixed order
// The scatter-add h'[r] = b[r] + sum_{j: pi(j) = r} D[j] h[j] adds every
// source that lands on row r.  No float atomics anywhere: the sum of each row
// runs in an order fixed by the map alone, so results are deterministic.
//
// Per dictionary entry the prep kernel stores one 64-bit word per index j:
//  - in-degree <= kMaxSrc everywhere (the usual case): the record of row j,
//    its sources in ascending order, one byte each (unused bytes name a row
//    that stays zero, or are masked by the in-degree), in-degree in the top
//    byte.  The step writes D .* h once and every row gathers its sources.
//  - some row above kMaxSrc (mtab = kFallback): the map's sorted form.  The
//    sources are ordered by (destination, source); bits 0-7 hold source j's
//    position in that order, bits 8-15 the last position of row j's run,
//    bit 16 says row j has a source, bit 17 that position j starts a run.
//    The step stores D[j] h[j] at j's position (a permutation, no
//    collisions), sums every run with a segmented scan across lanes, and each
//    row reads its run's total.
constexpr int kMaxSrc = 7;
constexpr unsigned kFallback = 255;

__device__ __forceinline__ int srt_pos(uint64_t w) { return (int)(w & 255u); }
__device__ __forceinline__ int srt_end(uint64_t w) { return (w >> 16) & 1u ? (int)((w >> 8) & 255u) : -1; }
__device__ __forceinline__ bool srt_start(uint64_t w) { return ((w >> 17) & 1u) != 0; }
__device__ __forceinline__ uint64_t srt_word(int pos, int end, bool has, bool start) {
    return (uint64_t)(pos & 255) | (uint64_t)(end & 255) << 8 | (uint64_t)(has ? 1 : 0) << 16 |
           (uint64_t)(start ? 1 : 0) << 17;
}

// Run totals of values in sorted order.  V holds N values, every row's
// sources contiguous; u = this lane's entries V[lane*SL + r], st[r] = whether
// position lane*SL + r starts a run, e[r] = the last position of the run of
// row lane*SL + r (-1: the row has no source).  Runs are summed by an
// in-lane pass and a segmented scan across lanes (a fixed order); V is
// overwritten.  Returns the run total of each of this lane's rows (0 when
// empty).  All 64 lanes must call it; act = lane holds entries.
template <int N, class E = float2>
__device__ __forceinline__ CV<Lay<N>::SL, E> run_totals(E* V, CV<Lay<N>::SL, E> u, const bool (&st)[Lay<N>::SL],
                                                        const int (&e)[Lay<N>::SL], int lane, bool act) {
    constexpr int SL = Lay<N>::SL;
    bool seen = false;
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        if (r > 0 && !st[r]) u.v[r] = cadd(u.v[r], u.v[r - 1]);
        seen |= st[r];
    }
    const uint64_t starts = __builtin_amdgcn_ballot_w64(act && seen);
    const E C = wave_seg_scan(u.v[SL - 1], starts, lane);
    if constexpr (SL == 1) {
        u.v[0] = C;
    } else {
        const E Cp = lane_up(C);
        bool head = false;
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            head |= st[r];
            if (!head) u.v[r] = cadd(u.v[r], Cp);
        }
    }
    wave_sync();
    if (act) st_cv<SL>(V, lane, u);
    wave_sync();
    CV<SL, E> tot = cv_zero<SL, E>();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            const E t = V[e[r] < 0 ? 0 : e[r]];
            tot.v[r] = e[r] < 0 ? ezero<E>() : t;
        }
    }
    return tot;
}

// h <- bt + P (Dt .* h) for a map given in sorted form (w = this lane's words
// of the entry).  V: N values of the wave's LDS scratch.
template <int N, class E = float2>
__device__ __forceinline__ void sorted_step(E* V, const uint64_t (&w)[Lay<N>::SL], CV<Lay<N>::SL, E>& h,
                                            const CV<Lay<N>::SL, E>& Dt, const CV<Lay<N>::SL, E>& bt, int lane,
                                            bool act) {
    constexpr int SL = Lay<N>::SL;
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) V[srt_pos(w[r])] = cmul(Dt.v[r], h.v[r]);
    }
    wave_sync();
    CV<SL, E> u = cv_zero<SL, E>();
    if (act) u = ld_cv<SL>(V, lane);
    bool st[SL];
    int e[SL];
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        st[r] = srt_start(w[r]);
        e[r] = srt_end(w[r]);
    }
    const CV<SL, E> tot = run_totals<N, E>(V, u, st, e, lane, act);
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) h.v[r] = cadd(bt.v[r], tot.v[r]);
    }
}

// Unused source bytes of a record: row N of the staged values (kept zero)
// when it fits in a byte; at N = 256 the in-degree byte masks them instead.
template <int N>
struct Sentinel {
    static constexpr bool kZeroRow = N <= 128;
    static constexpr unsigned kByte = N <= 128 ? (unsigned)N : 0u;
};

// Ranks of a map's sources in (destination, source) order.  pm: this lane's
// entries (source j = lane*SL + r goes to row pm[r]).  MT: SL tables of N
// 64-bit words in this wave's LDS scratch; table q collects, per row, the
// lanes whose slot q maps there (an atomic OR, whose result does not depend
// on the order of the ORs).  Returns, per source of this lane, its rank among
// the sources of its row (the lanes below it in the tables at its row, plus
// its own earlier slots with the same row), and per row of this lane its
// source count.
template <int N>
__device__ __forceinline__ void map_ranks(const IV<Lay<N>::SL>& pm, int lane, bool act,
                                          uint64_t* const (&MT)[Lay<N>::SL], int (&rank)[Lay<N>::SL],
                                          int (&cnt)[Lay<N>::SL]) {
    constexpr int SL = Lay<N>::SL;
    const uint64_t lt = (1ull << lane) - 1ull;
    wave_sync();
#pragma unroll
    for (int q = 0; q < SL; ++q)
        for (int i = lane; i < N; i += kWave) MT[q][i] = 0;
    wave_sync();
    if (act) {
#pragma unroll
        for (int q = 0; q < SL; ++q)
            __hip_atomic_fetch_or(MT[q] + pm.v[q], 1ull << lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
    }
    wave_sync();
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        int rk = 0, c = 0;
        if (act) {
#pragma unroll
            for (int q = 0; q < SL; ++q) {
                rk += __builtin_popcountll(MT[q][pm.v[r]] & lt);
                if (q < r) rk += pm.v[q] == pm.v[r] ? 1 : 0;
                c += __builtin_popcountll(MT[q][lane * SL + r]);
            }
        }
        rank[r] = rk;
        cnt[r] = c;
    }
}

// The sorted-form words (srt_word) of a map held in registers.  MT as for
// map_ranks; OFF: N ints and ST: N bytes of this wave's LDS scratch.
template <int N>
__device__ __forceinline__ void map_sorted_words(const IV<Lay<N>::SL>& pm, int lane, bool act,
                                                 uint64_t* const (&MT)[Lay<N>::SL], int* OFF, uint8_t* ST,
                                                 uint64_t (&w)[Lay<N>::SL]) {
    constexpr int SL = Lay<N>::SL;
    int rank[SL], cnt[SL];
    map_ranks<N>(pm, lane, act, MT, rank, cnt);
    int tot = 0;
#pragma unroll
    for (int r = 0; r < SL; ++r) tot += cnt[r];
    int off = wave_incl_scan_i(tot) - tot;  // first position of this lane's first row
    int ends[SL];
    wave_sync();
    for (int i = lane; i < N; i += kWave) ST[i] = 0;
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            OFF[lane * SL + r] = off;
            ends[r] = off + cnt[r] - 1;
            off += cnt[r];
        }
    }
    wave_sync();
    int pos[SL];
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            pos[r] = OFF[pm.v[r]] + rank[r];
            if (rank[r] == 0) ST[pos[r]] = 1;
        }
    }
    wave_sync();
#pragma unroll
    for (int r = 0; r < SL; ++r)
        w[r] = act ? srt_word(pos[r], ends[r], cnt[r] > 0, ST[lane * SL + r] != 0) : 0;
}

// h <- bt + P (Dt .* h) for a dictionary entry given by its prep words w
// (this lane's records, or its sorted form when cls == kFallback).  V: N + 1
// values of the wave's LDS scratch; V[N] must hold zero (N <= 128).  Every
// record's seven source slots are read; unused ones add zero.
template <int N>
__device__ __forceinline__ void table_step(float2* V, int cls, const uint64_t (&w)[Lay<N>::SL],
                                           CV<Lay<N>::SL>& h, const CV<Lay<N>::SL>& Dt,
                                           const CV<Lay<N>::SL>& bt, int lane, bool act) {
    constexpr int SL = Lay<N>::SL;
    if (cls == (int)kFallback) {
        sorted_step<N>(V, w, h, Dt, bt, lane, act);
        return;
    }
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) V[lane * SL + r] = cmul(Dt.v[r], h.v[r]);
    }
    wave_sync();
    if (act) {
#pragma unroll
        for (int r = 0; r < SL; ++r) {
            float2 acc = bt.v[r];
            const unsigned lo = (unsigned)w[r], hi = (unsigned)(w[r] >> 32);
#pragma unroll
            for (int m = 0; m < kMaxSrc; ++m) {
                const unsigned src = m < 4 ? (lo >> (8 * m)) & 255u : (hi >> (8 * (m - 4))) & 255u;
                float2 v = V[src];
                if constexpr (!Sentinel<N>::kZeroRow) v = m < (int)(hi >> 24) ? v : make_float2(0.f, 0.f);
                acc.x += v.x;
                acc.y += v.y;
            }
            h.v[r] = acc;
        }
    }
}

// acc += the sources M0 .. M1-1 of a record (V = the wave's staged values).
template <int M0, int M1, class E>
__device__ __forceinline__ void gather_rec_range(const E* V, uint64_t r, E& acc) {
    const unsigned lo = (unsigned)r, hi = (unsigned)(r >> 32);
#pragma unroll
    for (int m = M0; m < M1; ++m) {
        const unsigned src = m < 4 ? (lo >> (8 * m)) & 255u : (hi >> (8 * (m - 4))) & 255u;
        acc = cadd(acc, V[src]);
    }
}

// ------------------------------------------------------------------ cross-lane sums
// Cross-lane exchange primitives for the reduction below (VALU only, no LDS):
// permlane32/16 swaps trade the upper half of one register with the lower
// half of another across lanes l and l^32 (resp. l^16); DPP mirrors pair a
// lane with l^15 (16-lane row) and l^7 (8-lane half row); quad_perm pairs l^2
// and l^1.
__device__ __forceinline__ float dpp_f(float v, int ctrl) {
    switch (ctrl) {  // the control word must be a constant
        case 0x140: return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xf, 0xf, false));
        case 0x141: return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xf, 0xf, false));
        case 0x4e: return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4e, 0xf, 0xf, false));
        default: return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xb1, 0xf, 0xf, false));
    }
}

// Sum over the 64 lanes of each of T per-lane values v[t] (T a power of two
// <= 64), as a transpose-reduction: log2(T) halving exchanges in which each
// lane keeps half of its values (the half picked by one bit of its lane
// index), then plain butterflies.  Lane l ends with the total of value
// t = l / (64 / T).
template <int T>
__device__ __forceinline__ float transpose_sum(float (&v)[T], int lane) {
    int n = T;
#pragma unroll
    for (int lvl = 0; lvl < 6; ++lvl) {
        const int d = 32 >> lvl;
        if (n > 1) {
            const int h = n / 2;
#pragma unroll
            for (int i = 0; i < T / 2; ++i) {
                if (i < h) {
                    if (d >= 16) {
                        // lower lanes keep v[i] and receive the partner's v[i];
                        // upper lanes keep v[i+h] and receive the partner's v[i+h]
                        auto r = d == 32 ? __builtin_amdgcn_permlane32_swap(__float_as_uint(v[i]),
                                                                          __float_as_uint(v[i + h]), false, false)
                                         : __builtin_amdgcn_permlane16_swap(__float_as_uint(v[i]),
                                                                          __float_as_uint(v[i + h]), false, false);
                        v[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
                    } else {
                        const bool up = (lane & d) != 0;
                        const float send = up ? v[i] : v[i + h];
                        const float keep = up ? v[i + h] : v[i];
                        v[i] = keep + dpp_f(send, d == 8 ? 0x140 : d == 4 ? 0x141 : d == 2 ? 0x4e : 0xb1);
                    }
                }
            }
            n = h;
        } else {
            if (d >= 16) {
                auto r = d == 32 ? __builtin_amdgcn_permlane32_swap(__float_as_uint(v[0]), __float_as_uint(v[0]),
                                                                  false, false)
                                 : __builtin_amdgcn_permlane16_swap(__float_as_uint(v[0]), __float_as_uint(v[0]),
                                                                  false, false);
                v[0] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
            } else {
                v[0] += dpp_f(v[0], d == 8 ? 0x140 : d == 4 ? 0x141 : d == 2 ? 0x4e : 0xb1);
            }
        }
    }
    return v[0];
}

}  // namespace pdssm
