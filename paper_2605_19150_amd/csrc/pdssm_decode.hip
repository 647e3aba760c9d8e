// pdssm_decode.hip -- one step of the PD recurrence per sequence, for
// token-by-token inference (the constant-memory recurrent form of the
// model: the state h carries everything, Sec. 1 and App. E.2):
//
//   h'[r] = b[r] + sum_{j: pi(j) = r} D[j] h[j],   y = Re sum_n c[n] h'[n],
//   pi = pi[h, idx[b,h], :].
//
// The rows D, b, c come as complex64, bf16 (re, im) pairs or real fp32 (the
// real-valued model), widened to complex in registers as the scan kernels
// do; the state h stays complex64.
//
// One wave (one workgroup) per (batch, head) sequence; lane l owns entries
// l*SL .. l*SL+SL-1.  The scaled sources D[j] h[j] and the map are staged in
// LDS; each destination then adds its sources in ascending source order (a
// pass over the N sources with broadcast LDS reads, eight in flight), the
// order the scan kernels use, so colliding sources add deterministically.  The state may be updated in
// place: every lane has read its h entries before any lane writes.
#include "pdssm_decode.h"
#include "pdssm_device.h"

namespace pdssm {

namespace {

constexpr int kDecodeWaves = 1;  // one wave per workgroup: B*H workgroups spread over the CUs

// This lane's SL entries of row `row` (entries) of a [.., N] tensor in row format IO.
template <int SL, int IO>
__device__ __forceinline__ CV<SL> ld_row_io(const void* base, size_t row, int lane) {
    if constexpr (IO == kIoC64) {
        return ld_cv<SL>(static_cast<const float2*>(base) + row, lane);
    } else {
        const uint32_t* p = static_cast<const uint32_t*>(base) + row + (size_t)lane * SL;
        CV<SL> out;
#pragma unroll
        for (int s = 0; s < SL; ++s) out.v[s] = word_to_f2<IO>(p[s]);
        return out;
    }
}

template <int N, int IO>
__global__ __launch_bounds__(kDecodeWaves * 64) void k_decode(DecodeArgs a) {
    constexpr int SL = Lay<N>::SL, LANES = Lay<N>::LANES;
    __shared__ float2 vs[kDecodeWaves][N];
    __shared__ uint8_t ps[kDecodeWaves][N];
    const int wv = wave_id(), lane = lane_id();
    const int seq = blockIdx.x * kDecodeWaves + wv;
    if (seq >= a.B * a.H) return;
    const int hh = seq % a.H;
    const bool act = lane < LANES;
    const size_t row = (size_t)seq * N;
    float2* V = vs[wv];
    uint8_t* P = ps[wv];

    // the rows do not depend on the map: their loads go out first, then
    // idx and the map row it selects
    CV<SL> h = cv_zero<SL>(), D = cv_zero<SL>(), b = cv_zero<SL>(), c = cv_zero<SL>();
    if (act) {
        h = a.h_in ? ld_cv<SL>(a.h_in + row, lane) : cv_zero<SL>();
        D = ld_row_io<SL, IO>(a.D, row, lane);
        b = ld_row_io<SL, IO>(a.b, row, lane);
        c = ld_row_io<SL, IO>(a.c, row, lane);
    }
    int k = a.idx[seq];
    bool bad = (unsigned)k >= (unsigned)a.K;
    k = bad ? 0 : k;
    const int* pik = a.pi + ((size_t)hh * a.K + k) * N;
    IV<SL> p = {};
    if (act) {
        p = ld_iv<SL>(pik, lane);
        bad |= sanitize_map<N, SL>(p);
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            V[lane * SL + s] = cmul(D.v[s], h.v[s]);
            P[lane * SL + s] = (uint8_t)p.v[s];
        }
    }
    wave_sync();
    CV<SL> hn = b;
    if (act) {
#pragma unroll 8
        for (int j = 0; j < N; ++j) {
            const int r = P[j];
            const float2 v = V[j];
#pragma unroll
            for (int s = 0; s < SL; ++s)
                if (r == lane * SL + s) hn.v[s] = cadd(hn.v[s], v);
        }
    }
    float yl = 0.f;
#pragma unroll
    for (int s = 0; s < SL; ++s) yl += c.v[s].x * hn.v[s].x - c.v[s].y * hn.v[s].y;
    const float y = wave_sum_last(act ? yl : 0.f);
    if (act) st_cv<SL>(a.h_out + row, lane, hn);
    if (lane == kWave - 1) a.y[seq] = y;
    if (bad) report_index_error(a.status);
}

template <int N, int IO>
hipError_t decode_launch_io(const DecodeArgs& a, hipStream_t st) {
    const int nseq = a.B * a.H;
    auto kern = k_decode<N, IO>;
    hipLaunchKernelGGL(kern, dim3((nseq + kDecodeWaves - 1) / kDecodeWaves), dim3(kDecodeWaves * 64), 0, st, a);
    return hipGetLastError();
}

template <int N>
hipError_t decode_launch(const DecodeArgs& a, hipStream_t st) {
    switch (a.io) {
        case kIoC64: return decode_launch_io<N, kIoC64>(a, st);
        case kIoBf16: return decode_launch_io<N, kIoBf16>(a, st);
        case kIoReal: return decode_launch_io<N, kIoReal>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
    switch (a.N) {
        case 8: return decode_launch<8>(a, st);
        case 16: return decode_launch<16>(a, st);
        case 32: return decode_launch<32>(a, st);
        case 64: return decode_launch<64>(a, st);
        case 128: return decode_launch<128>(a, st);
        case 256: return decode_launch<256>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace pdssm
