// Cache append for the thin-key / full-value cache: the write that precedes
// decode. Token t of sequence b and KV head g is stored at cache position
// positions[b] + t: its r-entry key row (Sec. 2.4, Eq. 9) and its d_v-entry
// value row. With quantised keys each key row is quantised on the way in (the
// composition with quantisation the discussion in Sec. 6 proposes), with one
// fp32 scale per row, both steps in fp32 with IEEE division:
//  * E4M3: scale max|k| / 448 (1 for an all-zero row), code the OCP E4M3 of
//    k / scale rounded to nearest-even;
//  * 4-bit: scale max|k| / 7 (1 for an all-zero row), code k / scale rounded
//    half-to-even and clipped to [-7, 7], stored excess-8 (nibble code + 8, the
//    even entry in the low nibble).
//
// The kernel is a plain stream: every thread moves one 16-byte slice of a key or
// value row, read and written with non-temporal accesses. The R / 8 threads
// holding one key row are consecutive lanes, so the row maximum of the
// quantised paths is a butterfly over those lanes.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

#include <type_traits>

namespace tk {

namespace {

constexpr int kAppendThreads = 256;

// The new rows are read once and the cache rows written once, so both streams
// carry the non-temporal hint (no temporal reuse): with it the same accesses
// run about a tenth faster once neither stream can be served from a cache.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint4 load16_stream(const uint16_t* p) {
    const u32x4 v = __builtin_nontemporal_load((const u32x4*)p);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store16_stream(void* p, uint4 w) {
    u32x4 v;
    v[0] = w.x;
    v[1] = w.y;
    v[2] = w.z;
    v[3] = w.w;
    __builtin_nontemporal_store(v, (u32x4*)p);
}
__device__ __forceinline__ void store8_stream(void* p, uint32_t lo, uint32_t hi) {
    u32x2 v;
    v[0] = lo;
    v[1] = hi;
    __builtin_nontemporal_store(v, (u32x2*)p);
}
__device__ __forceinline__ void store4_stream(void* p, uint32_t w) { __builtin_nontemporal_store(w, (uint32_t*)p); }

// OCP E4M3FN encoding of an fp32 value, rounded to nearest-even: bias 7, three
// mantissa bits, subnormals with quantum 2^-9, largest finite 448, and no
// infinities (values past the largest finite, beyond the midpoint 464 to the
// next binade step, and NaN give the NaN code S.1111.111).
__device__ __forceinline__ uint32_t e4m3_rne(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t sign = (u >> 24) & 0x80u;
    const float a = fabsf(x);
    if (!(a <= 464.f)) return sign | 0x7fu;  // NaN, or above the last rounding midpoint
    if (a < 0.015625f) {                       // below 2^-6: multiples of 2^-9 (code 8 is 2^-6 itself)
        return sign | (uint32_t)__builtin_rintf(a * 512.f);
    }
    const uint32_t ua = u & 0x7fffffffu;
    int e = (int)(ua >> 23) - 127;               // -6 .. 8
    uint32_t q = ((ua & 0x7fffffu) | 0x800000u) >> 20;  // 1.mmm, implicit bit included
    const uint32_t rem = ua & 0xfffffu, half = 0x80000u;
    if (rem > half || (rem == half && (q & 1u))) ++q;
    if (q == 16u) {
        q = 8u;
        ++e;
    }
    const uint32_t code = ((uint32_t)(e + 7) << 3) | (q & 7u);
    return sign | (code > 0x7eu ? 0x7fu : code);
}

// Grid: x covers the 16-byte slices of one (sequence, KV head)'s new rows, y is
// the (sequence, KV head) pair, so a thread's token index is a shift.
template <int R, int DV, int KF, bool PAGED>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(const AppendParams p) {
    constexpr int KL = R / 8;   // threads per key row (8 entries each)
    constexpr int VL = DV / 8;  // threads per value row
    const int bg = blockIdx.y;
    const int b = bg / p.Hkv, g = bg - b * p.Hkv;
    const int start = p.pos[b];
    const int stride = gridDim.x * kAppendThreads;
    const int first = blockIdx.x * kAppendThreads + threadIdx.x;
    const uint16_t* kn = p.kn + (size_t)bg * p.T * R;
    const uint16_t* vn = p.vn + (size_t)bg * p.T * DV;

    // cache row of new token t, or -1 when it must not be written
    auto cache_row = [&](int t) -> long {
        const long pos = (long)start + t;
        if (pos < 0 || pos >= p.capacity) return -1;
        if constexpr (PAGED) {
            const int blk = p.table[(long)b * p.mb + (pos >> p.bs_log2)];
            if (blk < 0 || blk >= p.num_blocks) return -1;
            return (((long)blk * p.Hkv + g) << p.bs_log2) + (pos & ((1L << p.bs_log2) - 1));
        } else {
            return (long)bg * p.capacity + pos;
        }
    };

    // key rows: the KL threads of a row are consecutive lanes of one iteration
    // (the stride is a multiple of 64 and rows start at multiples of KL)
    for (int i = first; i < p.T * KL; i += stride) {
        const int t = i / KL, slice = i % KL;
        const long row = cache_row(t);
        const uint4 w = load16_stream(kn + (size_t)i * 8);
        if constexpr (KF != kKeyBF16) {
            const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
            float f[8];
            float amax = 0.f;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f[2 * j] = bf16lo(wd[j]);
                f[2 * j + 1] = bf16hi(wd[j]);
                amax = fmaxf(amax, fmaxf(fabsf(f[2 * j]), fabsf(f[2 * j + 1])));
            }
#pragma unroll
            for (int o = KL / 2; o >= 1; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o, 64));
            if constexpr (KF == kKeyE4M3) {
                const float scale = amax > 0.f ? amax / 448.f : 1.f;
                uint32_t code[2] = {0u, 0u};
#pragma unroll
                for (int j = 0; j < 8; ++j) code[j >> 2] |= e4m3_rne(f[j] / scale) << (8 * (j & 3));
                if (row >= 0) {
                    store8_stream(p.kc + row * R + slice * 8, code[0], code[1]);
                    if (slice == 0) p.ks[row] = scale;
                }
            } else {
                const float scale = amax > 0.f ? amax / 7.f : 1.f;
                uint32_t code = 0u;
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float c = fminf(fmaxf(__builtin_rintf(f[j] / scale), -7.f), 7.f);  // rint: half to even
                    code |= (uint32_t)((int)c + 8) << (4 * j);
                }
                if (row >= 0) {
                    store4_stream(p.kc + row * (R / 2) + slice * 4, code);
                    if (slice == 0) p.ks[row] = scale;
                }
            }
        } else {
            if (row >= 0) store16_stream(p.kc + (row * R + slice * 8) * 2, w);
        }
    }
    // value rows
    for (int i = first; i < p.T * VL; i += stride) {
        const long row = cache_row(i / VL);
        if (row >= 0) store16_stream(p.vc + row * DV + (i % VL) * 8, load16_stream(vn + (size_t)i * 8));
    }
}

template <int R, int DV>
hipError_t run(const AppendParams& p, int kf, bool paged, hipStream_t st) {
    const long work = (long)p.T * (DV / 8 > R / 8 ? DV / 8 : R / 8);
    long bx = (work + kAppendThreads - 1) / kAppendThreads;
    bx = bx < 1024 ? bx : 1024;  // grid-stride beyond that
    const dim3 grid((unsigned)bx, (unsigned)(p.B * p.Hkv)), block(kAppendThreads);
    auto launch = [&](auto kf_c) {
        constexpr int KF = decltype(kf_c)::value;
        if (paged)
            hipLaunchKernelGGL((append_kernel<R, DV, KF, true>), grid, block, 0, st, p);
        else
            hipLaunchKernelGGL((append_kernel<R, DV, KF, false>), grid, block, 0, st, p);
    };
    switch (kf) {
        case kKeyBF16: launch(std::integral_constant<int, kKeyBF16>{}); break;
        case kKeyE4M3: launch(std::integral_constant<int, kKeyE4M3>{}); break;
        case kKeyInt4: launch(std::integral_constant<int, kKeyInt4>{}); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int R>
hipError_t by_dv(const AppendParams& p, int DV, int kf, bool paged, hipStream_t st) {
    if (DV == 64) return run<R, 64>(p, kf, paged, st);
    if (DV == 128) return run<R, 128>(p, kf, paged, st);
    return hipErrorInvalidValue;
}

}  // namespace

tk_status launch_append(const AppendParams& p, int R, int DV, int kf, bool paged, hipStream_t st) {
    hipError_t e;
    switch (R) {
        case 16: e = by_dv<16>(p, DV, kf, paged, st); break;
        case 32: e = by_dv<32>(p, DV, kf, paged, st); break;
        case 64: e = by_dv<64>(p, DV, kf, paged, st); break;
        case 128: e = by_dv<128>(p, DV, kf, paged, st); break;
        default: return TK_ERR_UNSUPPORTED;
    }
    if (e == hipErrorInvalidValue) return TK_ERR_UNSUPPORTED;
    return e == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
