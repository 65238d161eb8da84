// Thin projections for factored keys (Sec. 2.3, Eq. 6-7): Y = X W for one
// projection of a layer, written head-major for the attention kernels.
//
// After a pretrained key projection is factored per KV head (W_K ~= A B) and B
// is absorbed into the query projection (W_Q' = W_Q B^T), the layer computes
// r-wide queries q' = x W_Q' and keys k' = x W_K' = x A for every token, and
// its full-width values v = x W_V. Each is a dense product of the token rows
// X [tokens, d_model] with a weight matrix whose columns are grouped by head.
// This kernel computes one such product on the bf16 matrix cores with fp32
// accumulation and stores the result straight into the [batch, head, token,
// width] layout that tk_attn_prefill and tk_cache_append read, so no separate
// transpose pass follows.
//
// The weight is passed transposed, Wt [n_heads * width, d_model] (one row per
// output column), so both operands of the product are contiguous along
// d_model. The tile computes C^T = Wt X^T: a lane of each 32x32 accumulator
// then holds four consecutive output columns of one token, which become one
// 8-byte store into the head-major output row.
#include "tk_device.hpp"
#include "tk_internal.hpp"

namespace tk {

namespace {

constexpr int kPBM = 128;  // tokens per workgroup tile
constexpr int kPBN = 128;  // output columns per workgroup tile
constexpr int kPBK = 64;   // d_model per k-tile (8 chunks of 8 bf16 per row)
constexpr int kPThreads = 256;
constexpr int kXcdCount = 8;
constexpr int kChunks = kPBM * kPBK / 8;  // 16-byte chunks of one operand tile (= kPBN * kPBK / 8)
constexpr int kPerThread = kChunks / kPThreads;
static_assert(kPBM == kPBN, "both operand tiles have the same shape");

struct ProjSmem {
    uint16_t w[2][kPBN * kPBK];  // Wt rows of the tile, XOR-swizzled 16-byte chunks
    uint16_t x[2][kPBM * kPBK];  // token rows of the tile, same swizzle
};

// element offset of chunk kc (0..7) of tile row r: chunks rotate by row so that
// the 32 rows one matrix-operand read touches spread over all LDS banks
__device__ __forceinline__ int sw(int r, int kc) { return r * kPBK + ((kc ^ (r & 7)) << 3); }

__global__ __launch_bounds__(kPThreads, 2) void project_kernel(const ProjectParams p) {
    __shared__ ProjSmem sm;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wn = wave >> 1, wm = wave & 1;  // this wave's 64x64 quarter of the tile
    // XCD-aware order: workgroups are dealt to the 8 XCDs round-robin; each XCD
    // takes a contiguous range of tiles, column tiles fastest, so the column
    // tiles of one token tile run on one XCD and share its rows through its L2
    const int per_xcd = (p.tiles + kXcdCount - 1) / kXcdCount;
    const int logical = (int)(blockIdx.x % kXcdCount) * per_xcd + (int)(blockIdx.x / kXcdCount);
    if (logical >= p.tiles) return;
    const int n_tiles = (p.N + kPBN - 1) / kPBN;
    const int n_base = (logical % n_tiles) * kPBN, m_base = (logical / n_tiles) * kPBM;
    const int col = lane & 31, half = lane >> 5;

    // chunk (row, kc) of each operand this thread stages, as byte offsets; rows
    // outside the matrix load zeros
    const uint16_t* wsrc[kPerThread];
    const uint16_t* xsrc[kPerThread];
    bool wok[kPerThread], xok[kPerThread];
    int soff[kPerThread];
#pragma unroll
    for (int i = 0; i < kPerThread; ++i) {
        const int c = tid + i * kPThreads, r = c >> 3, kc = c & 7;
        soff[i] = sw(r, kc);
        wok[i] = n_base + r < p.N;
        xok[i] = m_base + r < p.M;
        wsrc[i] = (const uint16_t*)p.wt + (size_t)(wok[i] ? n_base + r : 0) * p.K + kc * 8;
        xsrc[i] = (const uint16_t*)p.x + (size_t)(xok[i] ? m_base + r : 0) * p.K + kc * 8;
    }
    uint4 wreg[kPerThread], xreg[kPerThread];
    auto load = [&](int k0) {
#pragma unroll
        for (int i = 0; i < kPerThread; ++i) {
            const int kk = k0 + (((tid + i * kPThreads) & 7) << 3);
            wreg[i] = (wok[i] && kk < p.K) ? *(const uint4*)(wsrc[i] + k0) : make_uint4(0, 0, 0, 0);
            xreg[i] = (xok[i] && kk < p.K) ? *(const uint4*)(xsrc[i] + k0) : make_uint4(0, 0, 0, 0);
        }
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int i = 0; i < kPerThread; ++i) {
            *(uint4*)(sm.w[buf] + soff[i]) = wreg[i];
            *(uint4*)(sm.x[buf] + soff[i]) = xreg[i];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    const int nk = (p.K + kPBK - 1) / kPBK;
    load(0);
    stash(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load((kt + 1) * kPBK);
#pragma unroll
        for (int ks = 0; ks < kPBK / 16; ++ks) {
            const int kc = 2 * ks + half;
            bf16x8 a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int r = wn * 64 + i * 32 + col;
                a[i] = *(const bf16x8*)(sm.w[buf] + sw(r, kc));
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int r = wm * 64 + j * 32 + col;
                b[j] = *(const bf16x8*)(sm.x[buf] + sw(r, kc));
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) stash(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: lane (col, half) of block (i, j) holds output columns
    // n0 + 8 g + 4 half + 0..3 (g = 0..3) of token m0 + col, rounded to bf16 and
    // stored as 8 bytes into Y[b, h, s, w .. w + 3]
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int m = m_base + wm * 64 + j * 32 + col;
        if (m >= p.M) continue;
        const int bb = m / p.S, s = m - bb * p.S;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n = n_base + wn * 64 + i * 32 + 8 * g + 4 * half;
                if (n >= p.N) continue;
                const int h = n / p.width, w = n - h * p.width;
                uint2 v;
                v.x = pack_bf16(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                v.y = pack_bf16(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                *(uint2*)((uint16_t*)p.y + (((size_t)bb * p.heads + h) * p.S + s) * p.width + w) = v;
            }
        }
    }
}

}  // namespace

long project_tiles(long M, long N) { return ((M + kPBM - 1) / kPBM) * ((N + kPBN - 1) / kPBN); }

tk_status launch_project(const ProjectParams& p, hipStream_t st) {
    const long launched = ((long)p.tiles + kXcdCount - 1) / kXcdCount * kXcdCount;
    hipLaunchKernelGGL(project_kernel, dim3((unsigned)launched), dim3(kPThreads), 0, st, p);
    return hipGetLastError() == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
