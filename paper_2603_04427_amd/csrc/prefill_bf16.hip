// Thin-key causal prefill attention for gfx950, bf16 inputs, fp32 accumulation.
//
// Prefill is compute-bound (the paper's prefill-roofline appendix): per visible
// (query, key) pair it does 2r FLOPs of selection and 2 d_v FLOPs of value
// transfer, with r < d_v for thin keys. Both products run on the bf16 matrix
// cores (v_mfma_f32_32x32x16_bf16); the softmax runs on the vector ALUs.
//
// Work decomposition
//  * A workgroup is 4 waves. Wave w owns 32 query rows of one query head; the
//    workgroup covers HPW = gcd(G, 4) heads of one KV group and 4 / HPW blocks
//    of 32 rows, so every K/V tile staged in LDS serves 4 waves.
//  * Key tiles are 64 keys, double-buffered in LDS: K rows as they are in
//    memory (r wide, padded by 16 bytes), V transposed to [d_v][64] with the
//    keys of each 16-key group permuted so that one 16-byte LDS read yields a
//    lane's operand for the value product. The transpose happens in registers
//    (byte permutes) between the global load and the LDS store.
//  * Scores are computed transposed, S^T = K Q^T (keys along the MFMA rows,
//    queries along the columns): each lane then holds 16 keys of one query per
//    32-key block, so the row maximum and row sum are in-lane except for one
//    exchange between the two 32-lane halves, and P^T leaves the accumulators
//    already in the B-operand layout of O^T = V^T P^T.
//  * Online softmax in the log2 domain (scale * log2(e) applied in fp32 by one
//    FMA), with a lazy rescale: the running reference maximum moves only when
//    some row's maximum exceeds it by more than 8 (a factor of 256), so most
//    tiles skip rescaling the d_v x 32 accumulator.
//  * Causal masking is applied only on tiles that cross a wave's diagonal;
//    tiles entirely above it are skipped; query blocks are issued heaviest
//    first.
#include "tk_device.hpp"
#include "tk_internal.hpp"

#include <math.h>

namespace tk {

namespace {

constexpr int kThreads = 256;
constexpr int kBN = 64;          // keys per tile
constexpr int kVtStride = kBN + 8;  // bf16 elements per transposed V row (16-byte pad)

__host__ __device__ constexpr int gcd4(int g) { return (g % 4 == 0) ? 4 : (g % 2 == 0 ? 2 : 1); }

// Position of key k (0..63) inside a transposed V row: within each group of 16
// keys, k = 8a + 4b + c is stored at 8b + 4a + c.
__device__ __forceinline__ int vt_pos(int k) {
    const int a = (k >> 3) & 1, bb = (k >> 2) & 1, c = k & 3;
    return (k & ~15) + 8 * bb + 4 * a + c;
}

template <int R, int DV>
struct Smem {
    static constexpr int kStride = R + 8;  // bf16 elements per K row in LDS
    uint16_t k[2][kBN * kStride];
    uint16_t vt[2][DV * kVtStride];
};

template <int R, int DV>
struct TileRegs {
    static constexpr int kChunks = kBN * R / 8;                       // 16-byte K chunks per tile
    static constexpr int kLoads = (kChunks + kThreads - 1) / kThreads;  // per thread
    uint4 k[kLoads];
    uint4 v[4];
};

template <int R, int DV>
__device__ __forceinline__ void load_tile(TileRegs<R, DV>& t, const uint16_t* kg, const uint16_t* vg, int base,
                                          int Sk, int tid) {
    constexpr int CPR = R / 8;  // 16-byte chunks per K row
#pragma unroll
    for (int i = 0; i < TileRegs<R, DV>::kLoads; ++i) {
        const int c = tid + i * kThreads;
        const int row = c / CPR, part = c % CPR;
        const bool ok = c < TileRegs<R, DV>::kChunks && base + row < Sk;
        t.k[i] = ok ? *(const uint4*)(kg + (size_t)(base + row) * R + part * 8) : make_uint4(0, 0, 0, 0);
    }
    // V: thread -> (key quad kq, 8-column chunk dc)
    const int kq = tid & 15, dc = tid >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int key = base + 4 * kq + i;
        const bool ok = dc < DV / 8 && key < Sk;
        t.v[i] = ok ? *(const uint4*)(vg + (size_t)key * DV + dc * 8) : make_uint4(0, 0, 0, 0);
    }
}

template <int R, int DV>
__device__ __forceinline__ void store_tile(const TileRegs<R, DV>& t, uint16_t* ks, uint16_t* vts, int tid) {
    constexpr int CPR = R / 8;
    constexpr int KS = Smem<R, DV>::kStride;
#pragma unroll
    for (int i = 0; i < TileRegs<R, DV>::kLoads; ++i) {
        const int c = tid + i * kThreads;
        if (c < TileRegs<R, DV>::kChunks) {
            const int row = c / CPR, part = c % CPR;
            *(uint4*)(ks + row * KS + part * 8) = t.k[i];
        }
    }
    const int kq = tid & 15, dc = tid >> 4;
    if (dc < DV / 8) {
        const int pos = vt_pos(4 * kq);
        const uint32_t x0[4] = {t.v[0].x, t.v[0].y, t.v[0].z, t.v[0].w};
        const uint32_t x1[4] = {t.v[1].x, t.v[1].y, t.v[1].z, t.v[1].w};
        const uint32_t x2[4] = {t.v[2].x, t.v[2].y, t.v[2].z, t.v[2].w};
        const uint32_t x3[4] = {t.v[3].x, t.v[3].y, t.v[3].z, t.v[3].w};
#pragma unroll
        for (int pr = 0; pr < 4; ++pr) {
            // columns 2pr (low halves) and 2pr+1 (high halves) of the 4 keys
            uint2 lo, hi;
            lo.x = __builtin_amdgcn_perm(x1[pr], x0[pr], 0x05040100u);
            lo.y = __builtin_amdgcn_perm(x3[pr], x2[pr], 0x05040100u);
            hi.x = __builtin_amdgcn_perm(x1[pr], x0[pr], 0x07060302u);
            hi.y = __builtin_amdgcn_perm(x3[pr], x2[pr], 0x07060302u);
            const int d = dc * 8 + 2 * pr;
            *(uint2*)(vts + d * kVtStride + pos) = lo;
            *(uint2*)(vts + (d + 1) * kVtStride + pos) = hi;
        }
    }
}

}  // namespace

template <int R, int DV>
__global__ __launch_bounds__(kThreads, 2) void prefill_bf16_kernel(const PrefillParams p) {
    constexpr int KSTEPS = R / 16;  // MFMA K-steps of the score product
    constexpr int DBLK = DV / 32;   // 32-row blocks of O^T
    constexpr int KS = Smem<R, DV>::kStride;
    __shared__ Smem<R, DV> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, col = lane & 31;

    const int HPW = gcd4(p.G);
    const int RB = 4 / HPW;
    const int BM = 32 * RB;
    const int nqb = (p.Sq + BM - 1) / BM;
    const int qb = p.causal ? nqb - 1 - (int)blockIdx.x : (int)blockIdx.x;  // heaviest first
    const int groups_per_kv = p.G / HPW;
    const int g = blockIdx.y / groups_per_kv;
    const int h = g * p.G + (blockIdx.y % groups_per_kv) * HPW + wave % HPW;
    const int b = blockIdx.z;
    const int q0 = qb * BM;                     // first row of the workgroup
    const int qw0 = q0 + (wave / HPW) * 32;     // first row of this wave
    const int off = p.Sk - p.Sq;                // bottom-right causal alignment

    const uint16_t* qg = (const uint16_t*)p.q + ((size_t)b * p.Hq + h) * p.Sq * R;
    const uint16_t* kg = (const uint16_t*)p.k + ((size_t)b * p.Hkv + g) * p.Sk * R;
    const uint16_t* vg = (const uint16_t*)p.v + ((size_t)b * p.Hkv + g) * p.Sk * DV;
    uint16_t* og = (uint16_t*)p.o + ((size_t)b * p.Hq + h) * p.Sq * DV;

    // Q^T operand: query row qw0 + col, dims 16m + 8 half .. +7
    const int qrow = qw0 + col;
    bf16x8 qreg[KSTEPS];
#pragma unroll
    for (int m = 0; m < KSTEPS; ++m) {
        uint4 w = qrow < p.Sq ? *(const uint4*)(qg + (size_t)qrow * R + 16 * m + 8 * half) : make_uint4(0, 0, 0, 0);
        qreg[m] = __builtin_bit_cast(bf16x8, w);
    }

    int key_end = p.Sk;
    if (p.causal) {
        const int last = q0 + BM - 1 + off + 1;
        key_end = last < key_end ? last : key_end;
    }
    const int ntiles = (key_end + kBN - 1) / kBN;
    // last key any row of this wave may see
    const int wave_last_key = p.causal ? qw0 + 31 + off : p.Sk - 1;

    f32x16 o[DBLK];
#pragma unroll
    for (int d = 0; d < DBLK; ++d)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[d][v] = 0.f;
    float m_ref = -INFINITY;  // running reference maximum (log2 domain) of this lane's row
    float lsum = 0.f;         // this lane's half of the row sum
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
            const uint16_t* ks = sm.k[cur];
            const uint16_t* vts = sm.vt[cur];
            // ---- S^T = K Q^T for the two 32-key blocks
            f32x16 s[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
                for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
#pragma unroll
                for (int m = 0; m < KSTEPS; ++m) {
                    const bf16x8 a = *(const bf16x8*)(ks + (kb * 32 + col) * KS + 16 * m + 8 * half);
                    s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[m], s[kb], 0, 0, 0);
                }
            }
            // ---- causal / ragged-tail mask, only where the tile crosses it
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
            // ---- row maximum (in-lane over 32 keys, then across the halves)
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
            // ---- probabilities -> bf16 B operands of O^T = V^T P^T
            bf16x8 pb[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float p0 = exp2_fast(fmaf(s[q >> 1][8 * (q & 1) + 2 * i], c, -m_ref));
                    const float p1 = exp2_fast(fmaf(s[q >> 1][8 * (q & 1) + 2 * i + 1], c, -m_ref));
                    w[i] = pack_bf16(p0, p1);
                    lsum = add_bf16_pair(w[i], lsum);
                }
                pb[q] = __builtin_bit_cast(bf16x8, make_uint4(w[0], w[1], w[2], w[3]));
            }
            // ---- O^T += V^T P^T
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int d = 0; d < DBLK; ++d) {
                    const bf16x8 a = *(const bf16x8*)(vts + (d * 32 + col) * kVtStride + 16 * q + 8 * half);
                    o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[q], o[d], 0, 0, 0);
                }
        }

        if (t + 1 < ntiles) store_tile<R, DV>(regs, sm.k[cur ^ 1], sm.vt[cur ^ 1], tid);
        __syncthreads();
    }

    // ---- epilogue: normalise and store bf16 rows
    const float ltot = lsum + __shfl_xor(lsum, 32);
    const float inv = 1.f / ltot;
    if (qrow < p.Sq) {
        uint16_t* orow = og + (size_t)qrow * DV;
#pragma unroll
        for (int d = 0; d < DBLK; ++d)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                uint2 w;
                w.x = pack_bf16(o[d][4 * j] * inv, o[d][4 * j + 1] * inv);
                w.y = pack_bf16(o[d][4 * j + 2] * inv, o[d][4 * j + 3] * inv);
                *(uint2*)(orow + d * 32 + 8 * j + 4 * half) = w;
            }
    }
}

template <int R, int DV>
static hipError_t run(const PrefillParams& p, hipStream_t st) {
    const int HPW = gcd4(p.G);
    const int BM = 32 * (4 / HPW);
    dim3 grid((p.Sq + BM - 1) / BM, p.Hkv * (p.G / HPW), p.B);
    hipLaunchKernelGGL((prefill_bf16_kernel<R, DV>), grid, dim3(kThreads), 0, st, p);
    return hipGetLastError();
}

template <int R>
static hipError_t by_dv(const PrefillParams& p, int DV, hipStream_t st) {
    if (DV == 64) return run<R, 64>(p, st);
    if (DV == 128) return run<R, 128>(p, st);
    return hipErrorInvalidValue;
}

tk_status launch_prefill_bf16(const PrefillParams& p, int R, int DV, hipStream_t st) {
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
