// Thin-key prefill attention for gfx950 with fp32 inputs and fp32 matrix cores
// (v_mfma_f32_32x32x2f32), for callers that need fp32 accuracy (bf16 operands
// would not hold a 1e-4 error bound).
//
// Same decomposition as the bf16 kernel: 4 waves of 32 query rows, 64-key tiles
// double-buffered in LDS, transposed scores S^T = K Q^T so each lane owns one
// query column, and O^T = V^T P^T. With K = 2 per instruction each 32-lane half
// contributes one contraction index per step, so:
//  * the score product walks r in R/2 steps, lane half h covering dims
//    [h R/2, (h+1) R/2) (contiguous in the K row, read 16 bytes at a time);
//  * the value product walks the 32 keys of a block in 16 steps, lane half h
//    supplying the key that its accumulator register already holds, so P^T is
//    used in place with no repacking. V is stored transposed ([d_v][64] fp32,
//    natural key order) so four consecutive steps' operands are one 16-byte read.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

namespace tk {

namespace {

constexpr int kThreads = 256;
constexpr int kBN = 64;
constexpr int kVtStride = kBN + 4;  // floats per transposed V row (16-byte pad)

__host__ __device__ constexpr int gcd4(int g) { return (g % 4 == 0) ? 4 : (g % 2 == 0 ? 2 : 1); }

template <int R, int DV>
struct Smem {
    static constexpr int kStride = R + 4;  // floats per K row in LDS
    float k[2][kBN * kStride];
    float vt[2][DV * kVtStride];
};

template <int R, int DV>
struct TileRegs {
    static constexpr int kKChunks = kBN * R / 4;  // 16-byte K chunks per tile
    static constexpr int kKLoads = (kKChunks + kThreads - 1) / kThreads;
    static constexpr int kVQuads = (kBN / 4) * (DV / 4);  // 4 keys x 4 columns per quad
    static constexpr int kVLoads = (kVQuads + kThreads - 1) / kThreads;
    float4 k[kKLoads];
    float4 v[kVLoads][4];
};

template <int R, int DV>
__device__ __forceinline__ void load_tile(TileRegs<R, DV>& t, const float* kg, const float* vg, int base, int Sk,
                                          int tid) {
    constexpr int CPR = R / 4;
#pragma unroll
    for (int i = 0; i < TileRegs<R, DV>::kKLoads; ++i) {
        const int c = tid + i * kThreads;
        const int row = c / CPR, part = c % CPR;
        const bool ok = c < TileRegs<R, DV>::kKChunks && base + row < Sk;
        t.k[i] = ok ? *(const float4*)(kg + (size_t)(base + row) * R + part * 4) : make_float4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < TileRegs<R, DV>::kVLoads; ++i) {
        const int qd = tid + i * kThreads;
        const int kq = qd % (kBN / 4), dc = qd / (kBN / 4);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int key = base + 4 * kq + j;
            const bool ok = qd < TileRegs<R, DV>::kVQuads && key < Sk;
            t.v[i][j] = ok ? *(const float4*)(vg + (size_t)key * DV + dc * 4) : make_float4(0, 0, 0, 0);
        }
    }
}

template <int R, int DV>
__device__ __forceinline__ void store_tile(const TileRegs<R, DV>& t, float* ks, float* vts, int tid) {
    constexpr int CPR = R / 4;
    constexpr int KS = Smem<R, DV>::kStride;
#pragma unroll
    for (int i = 0; i < TileRegs<R, DV>::kKLoads; ++i) {
        const int c = tid + i * kThreads;
        if (c < TileRegs<R, DV>::kKChunks) {
            const int row = c / CPR, part = c % CPR;
            *(float4*)(ks + row * KS + part * 4) = t.k[i];
        }
    }
#pragma unroll
    for (int i = 0; i < TileRegs<R, DV>::kVLoads; ++i) {
        const int qd = tid + i * kThreads;
        if (qd < TileRegs<R, DV>::kVQuads) {
            const int kq = qd % (kBN / 4), dc = qd / (kBN / 4);
            const float4* x = t.v[i];
            // 4 keys x 4 columns -> 4 rows of V^T, 4 consecutive keys each
            *(float4*)(vts + (dc * 4 + 0) * kVtStride + 4 * kq) = make_float4(x[0].x, x[1].x, x[2].x, x[3].x);
            *(float4*)(vts + (dc * 4 + 1) * kVtStride + 4 * kq) = make_float4(x[0].y, x[1].y, x[2].y, x[3].y);
            *(float4*)(vts + (dc * 4 + 2) * kVtStride + 4 * kq) = make_float4(x[0].z, x[1].z, x[2].z, x[3].z);
            *(float4*)(vts + (dc * 4 + 3) * kVtStride + 4 * kq) = make_float4(x[0].w, x[1].w, x[2].w, x[3].w);
        }
    }
}

}  // namespace

template <int R, int DV>
__global__ __launch_bounds__(kThreads, 1) void prefill_f32_kernel(const PrefillParams p) {
    constexpr int HR = R / 2;      // score-product steps (dims per lane half)
    constexpr int DBLK = DV / 32;
    constexpr int KS = Smem<R, DV>::kStride;
    __shared__ Smem<R, DV> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, col = lane & 31;

    const int HPW = gcd4(p.G);
    const int RB = 4 / HPW;
    const int BM = 32 * RB;
    const int nqb = (p.Sq + BM - 1) / BM;
    const int qb = p.causal ? nqb - 1 - (int)blockIdx.x : (int)blockIdx.x;
    const int groups_per_kv = p.G / HPW;
    const int g = blockIdx.y / groups_per_kv;
    const int h = g * p.G + (blockIdx.y % groups_per_kv) * HPW + wave % HPW;
    const int b = blockIdx.z;
    const int q0 = qb * BM;
    const int qw0 = q0 + (wave / HPW) * 32;
    const int off = p.Sk - p.Sq;

    const float* qg = (const float*)p.q + ((size_t)b * p.Hq + h) * p.Sq * R;
    const float* kg = (const float*)p.k + ((size_t)b * p.Hkv + g) * p.Sk * R;
    const float* vg = (const float*)p.v + ((size_t)b * p.Hkv + g) * p.Sk * DV;
    float* og = (float*)p.o + ((size_t)b * p.Hq + h) * p.Sq * DV;

    const int qrow = qw0 + col;
    float qreg[HR];
#pragma unroll
    for (int s = 0; s < HR; ++s) qreg[s] = qrow < p.Sq ? qg[(size_t)qrow * R + half * HR + s] : 0.f;

    int key_end = p.Sk;
    if (p.causal) {
        const int last = q0 + BM - 1 + off + 1;
        key_end = last < key_end ? last : key_end;
    }
    const int ntiles = (key_end + kBN - 1) / kBN;
    const int wave_last_key = p.causal ? qw0 + 31 + off : p.Sk - 1;

    f32x16 o[DBLK];
#pragma unroll
    for (int d = 0; d < DBLK; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[d][v] = 0.f;
    float m_ref = -INFINITY;
    float lsum = 0.f;
    const float c = p.qscale;

    TileRegs<R, DV> regs;
    load_tile<R, DV>(regs, kg, vg, 0, p.Sk, tid);
    store_tile<R, DV>(regs, sm.k[0], sm.vt[0], tid);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const int cur = t & 1;
        const int base = t * kBN;
        if (t + 1 < ntiles) load_tile<R, DV>(regs, kg, vg, base + kBN, p.Sk, tid);

        if (base <= wave_last_key) {
            const float* ks = sm.k[cur];
            const float* vts = sm.vt[cur];
            f32x16 s[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
                const float* krow = ks + (kb * 32 + col) * KS + half * HR;
#pragma unroll
                for (int s4 = 0; s4 < HR; s4 += 4) {
                    const float4 a = *(const float4*)(krow + s4);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, qreg[s4 + 0], s[kb], 0, 0, 0);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, qreg[s4 + 1], s[kb], 0, 0, 0);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, qreg[s4 + 2], s[kb], 0, 0, 0);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, qreg[s4 + 3], s[kb], 0, 0, 0);
                }
            }
            const bool needs_mask = (p.causal && base + kBN - 1 > qw0 + off) || base + kBN > p.Sk;
            if (needs_mask) {
                const int limit = p.causal ? qrow + off : p.Sk - 1;
                const int lim = limit < p.Sk - 1 ? limit : p.Sk - 1;
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int key = base + kb * 32 + 8 * (v >> 2) + 4 * half + (v & 3);
                        if (key > lim) s[kb][v] = -INFINITY;
                    }
            }
            float mx = s[0][0];
#pragma unroll
            for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[0][v]);
#pragma unroll
            for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[1][v]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float mx2 = mx * c;
            // each row moves its own reference only; the branch is taken by the
            // whole wave when any row needs it
            const bool need = mx2 > m_ref + 8.f;
            if (__any(need)) {
                const float alpha = need ? exp2_fast(m_ref - mx2) : 1.f;
                m_ref = need ? mx2 : m_ref;
                lsum *= alpha;
#pragma unroll
                for (int d = 0; d < DBLK; ++d)
#pragma unroll
                    for (int v = 0; v < 16; ++v) o[d][v] *= alpha;
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    s[kb][v] = exp2_fast(fmaf(s[kb][v], c, -m_ref));
                    lsum += s[kb][v];
                }
            // O^T += V^T P^T, one key per lane half per step
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int d = 0; d < DBLK; ++d) {
                    const float* vrow = vts + (d * 32 + col) * kVtStride + kb * 32 + 4 * half;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const float4 a = *(const float4*)(vrow + 8 * j);
                        o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, s[kb][4 * j + 0], o[d], 0, 0, 0);
                        o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, s[kb][4 * j + 1], o[d], 0, 0, 0);
                        o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, s[kb][4 * j + 2], o[d], 0, 0, 0);
                        o[d] = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, s[kb][4 * j + 3], o[d], 0, 0, 0);
                    }
                }
        }

        if (t + 1 < ntiles) store_tile<R, DV>(regs, sm.k[cur ^ 1], sm.vt[cur ^ 1], tid);
        __syncthreads();
    }

    const float ltot = lsum + __shfl_xor(lsum, 32);
    const float inv = 1.f / ltot;
    if (qrow < p.Sq) {
        float* orow = og + (size_t)qrow * DV;
#pragma unroll
        for (int d = 0; d < DBLK; ++d)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                *(float4*)(orow + d * 32 + 8 * j + 4 * half) =
                    make_float4(o[d][4 * j] * inv, o[d][4 * j + 1] * inv, o[d][4 * j + 2] * inv, o[d][4 * j + 3] * inv);
    }
}

template <int R, int DV>
static hipError_t run(const PrefillParams& p, hipStream_t st) {
    const int HPW = gcd4(p.G);
    const int BM = 32 * (4 / HPW);
    dim3 grid((p.Sq + BM - 1) / BM, p.Hkv * (p.G / HPW), p.B);
    hipLaunchKernelGGL((prefill_f32_kernel<R, DV>), grid, dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

template <int R>
static hipError_t by_dv(const PrefillParams& p, int DV, hipStream_t st) {
    if (DV == 64) return run<R, 64>(p, st);
    if (DV == 128) return run<R, 128>(p, st);
    return hipErrorInvalidValue;
}

tk_status launch_prefill_f32(const PrefillParams& p, int R, int DV, hipStream_t st) {
    hipError_t e;
    switch (R) {
        case 16: e = by_dv<16>(p, DV, st); break;
        case 32: e = by_dv<32>(p, DV, st); break;
        case 64: e = by_dv<64>(p, DV, st); break;
        case 128: e = by_dv<128>(p, DV, st); break;
        default: return TK_ERR_UNSUPPORTED;
    }
    if (e == hipErrorInvalidValue) return TK_ERR_UNSUPPORTED;
    return e == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
