// HIP kernels (gfx950, wave64) of the structured-dropout LSTM training step.
//
// Every product runs on MFMA 16x16x32 tiles (bf16 inputs with fp32
// accumulation; the fp32 path issues the fp32 MFMA).  Operands are gathered
// through the keep lists while they are loaded, so the dropped rows of a
// contraction are never read or multiplied (compact mode).  In dense mode
// the keep lists are the identity and the mask zeroes the dropped operands.
//
// Layouts (B = batch, BP = B rounded up to 32, G = 4H):
//   row-major activations [B][K]        forward products (gather along K)
//   transposed activations [K][BP]      weight gradients (contiguous in b)
//   DA [B][G] fragment-major            backward products (one 1 KB block per A fragment)
//   DA^T [G][BP]                        weight gradients
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <stdlib.h>
#include <string.h>

#include <vector>

#include "device.h"
#include "kernels.h"
#include "../../include/lstm_sd.h"

namespace lsd {

// ---------------------------------------------------------------------------
// Vector loads of 4 consecutive elements (8-byte aligned for bf16, 16 for f32)
__device__ __forceinline__ void ld4(const bf16* p, bf16* o) {
    const uint2 v = *(const uint2*)p;
    o[0] = (bf16)(v.x & 0xffffu); o[1] = (bf16)(v.x >> 16);
    o[2] = (bf16)(v.y & 0xffffu); o[3] = (bf16)(v.y >> 16);
}
__device__ __forceinline__ void ld4(const float* p, float* o) {
    const float4 v = *(const float4*)p;
    o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
}
template <typename T>
__device__ __forceinline__ void zero4(T* o) {
    o[0] = o[1] = o[2] = o[3] = zero_val<T>();
}
// Workgroups are dealt to the 8 XCDs round-robin (linear workgroup id i runs
// on XCD i % 8).  xcd_tile maps the x index of a grid whose x size is a
// multiple of 8 to a logical tile so that every XCD owns one contiguous range
// of tiles (and its L2 keeps the matching slice of the weights); -1 = idle.
constexpr int NXCD = 8;
constexpr int NSEG = 16;                   // keep-list segments: slice x of 8 is segments 2x, 2x+1
__device__ __forceinline__ int xcd_tile(int bx, int ntiles) {
    const int per = (ntiles + NXCD - 1) / NXCD;
    const int x = bx % NXCD, i = bx / NXCD;
    const int tile = x * per + i;
    return (i < per && tile < ntiles) ? tile : -1;
}
// First neuron of slice x of a K-neuron site (slices of floor(x*K/8)).
__device__ __forceinline__ int slice_start(int x, int K) { return (x * K) / NXCD; }
__device__ __forceinline__ int seg_start(int x, int K) { return (x * K) / NSEG; }   // seg_start(2x) = slice_start(x)

// ---------------------------------------------------------------------------
// Masks (Sec. 3.1, Case-III) and their compaction into keep/drop lists.
// grid (T, sites), block 256.
__global__ void __launch_bounds__(256) k_mask_build(MaskArgs a) {
    const int t = blockIdx.x, s = blockIdx.y, tid = threadIdx.x;
    const int K = a.K[s];
    __shared__ uint8_t sm[LSTM_SD_MAX_K];
    __shared__ int kpre[LSTM_SD_MAX_K];        // kept entries before k (compact mode)
    __shared__ int wsum[4], wdrop[4];
    const size_t row = ((size_t)s * a.T + t) * a.kmax;
    uint8_t* mrow = a.mask + row;
    int32_t* krow = a.keep + row;
    int32_t* prow = a.pos + row;
    int32_t* drow = a.drop + row;
    int32_t* ksrow = a.kseg + ((size_t)s * a.T + t) * (NSEG + 1);
    int32_t* dsrow = a.dseg + ((size_t)s * a.T + t) * (NSEG + 1);
    if (a.generate) {
        const uint64_t thr = a.thr[s];
        for (int q = tid; q < (K + 3) / 4; q += blockDim.x) {
            u64x4 c;
            c.x[0] = (uint64_t)q;
            c.x[1] = a.fixed ? 0ull : (uint64_t)t;
            c.x[2] = (uint64_t)a.sid[s];
            c.x[3] = a.step;
            const u64x4 r = philox4x64_10(c, a.seed, 0ull);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int k = 4 * q + e;
                if (k < K) {
                    const uint8_t kept = (thr == 0 || r.x[e] >= thr) ? 1 : 0;
                    sm[k] = kept;
                    mrow[k] = kept;
                }
            }
        }
    } else {
        for (int k = tid; k < K; k += blockDim.x) sm[k] = mrow[k] ? 1 : 0;
    }
    __syncthreads();
    if (!a.compact) {
        for (int k = tid; k < K; k += blockDim.x) { krow[k] = k; prow[k] = k; }
        if (tid <= NSEG) {
            ksrow[tid] = seg_start(tid, K);
            dsrow[tid] = 0;
        }
        if (tid == 0) {
            a.count[(size_t)s * a.T + t] = K;
            a.dcount[(size_t)s * a.T + t] = 0;
        }
        return;
    }
    const int lane = tid & 63, w = tid >> 6;
    int base = 0, dbase = 0;
    for (int k0 = 0; k0 < K; k0 += 256) {
        const int k = k0 + tid;
        const int f = (k < K) ? sm[k] : 0;
        const int g = (k < K) ? 1 - f : 0;
        const unsigned long long bal = __ballot(f);
        const unsigned long long dbal = __ballot(g);
        const unsigned long long below = (1ull << lane) - 1ull;
        const int pre = __popcll(bal & below), dpre = __popcll(dbal & below);
        if (lane == 0) { wsum[w] = __popcll(bal); wdrop[w] = __popcll(dbal); }
        __syncthreads();
        int off = base, doff = dbase;
        for (int i = 0; i < w; ++i) { off += wsum[i]; doff += wdrop[i]; }
        const int tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
        const int dtot = wdrop[0] + wdrop[1] + wdrop[2] + wdrop[3];
        if (k < K) {
            if (f) { krow[off + pre] = k; prow[k] = off + pre; }
            else { drow[doff + dpre] = k; prow[k] = -1; }
            kpre[k] = off + pre;
        }
        base += tot;
        dbase += dtot;
        __syncthreads();
    }
    // segment x starts at entry seg_start(x, K): its keep-list range starts
    // at the number of kept entries before it, its drop-list range at the
    // number dropped before it
    if (tid < NSEG) {
        const int sx = seg_start(tid, K);
        ksrow[tid] = kpre[sx];
        dsrow[tid] = sx - kpre[sx];
    }
    if (tid == 0) {
        a.count[(size_t)s * a.T + t] = base;
        a.dcount[(size_t)s * a.T + t] = dbase;
        ksrow[NSEG] = base;
        dsrow[NSEG] = dbase;
    }
}

// ---------------------------------------------------------------------------
// src [N][B][K] -> dst [N][K][BP], zero rows b in [B, BP); two such jobs
// (matrices z < n1 from the first, the others from the second) in one grid,
// and, with n_init > 0, the forward pass's initialisation in slice z = N.
// One workgroup (256 threads) of a grid (gx = ceil(max K/32), gy = BP/32,
// N (+1)): block (bx, by, bz).
template <typename T>
__device__ __forceinline__ void transpose_block(const TransArgs& a, int N, int bx, int by, int bz, int gx, int gy,
                                                T (*tile)[33]) {
    const int tid = threadIdx.x, tx = tid & 31, ty = tid >> 5;
    if (bz == N) {
        const long nb = (long)gx * gy, bi = (long)by * gx + bx;
        if (bi == 0) {
            for (int i = tid; i <= BAR_LINES * BAR_EXIT; i += 256) a.bar[BAR_PITCH * i] = 0u;
            if (tid == 0) {
                *a.err = 0;
                *(int*)((char*)a.err + (SYNC_STATUS_OFS - SYNC_ERR_OFS)) = 0;   // a new step's status
            }
        }
        for (long i = bi * 256 + tid; i < a.n_init; i += nb * 256) {
            a.hT[i] = to_f32<T>(((const T*)a.h0)[i]);
            a.cT[i] = a.c0[i];
        }
        return;
    }
    const bool second = bz >= a.n1;
    const int n = second ? bz - a.n1 : bz, K = second ? a.K2 : a.K;
    const int k0 = bx * 32, b0 = by * 32;
    if (k0 >= K) return;                       // (the whole workgroup)
    const T* src = (const T*)(second ? a.src2 : a.src) + (size_t)n * a.B * K;
    T* dst = (T*)(second ? a.dst2 : a.dst) + (size_t)n * K * a.BP;
    for (int i = ty; i < 32; i += 8) {
        const int b = b0 + i, k = k0 + tx;
        tile[i][tx] = (b < a.B && k < K) ? src[(size_t)b * K + k] : zero_val<T>();
    }
    __syncthreads();
    for (int i = ty; i < 32; i += 8) {
        const int k = k0 + i, b = b0 + tx;
        if (k < K) dst[(size_t)k * a.BP + b] = tile[tx][i];
    }
}

// ---------------------------------------------------------------------------
// Forward input product, all t (Eq. 1-4 first term; Sec. 3.2, FP input
// sparsity: the dropped columns of x and rows of W are skipped).
// grid (ceil(G/128) on the XCD mapping, T, ceil(B/32)), block 256.  A
// workgroup computes a 32-row x 128-column tile of Gx_t; wave w owns columns
// 32w .. 32w+31 (two 16-column MFMA tiles) for both 16-row tiles.  The
// contraction runs over the keep list of t in chunks of 32 kept rows: each
// chunk of W (32 gathered rows x 128 columns, loaded as whole row segments)
// and of X (32 rows x the 32 gathered columns) is staged in LDS, double
// buffered so that chunk i+1 is fetched while chunk i is multiplied.
// Columns past G read neighbouring (or, at the end, out-of-range = zero) W
// data and are never stored.
constexpr int FX_NB = 128, FX_MB = 32, FX_KC = 32, FX_LD = FX_KC + 8;
constexpr int FX_WLD = FX_NB + 8;

template <typename T, bool DENSE>
__global__ void __launch_bounds__(256) k_fx(FxArgs a) {
    constexpr uint32_t ES = sizeof(T);
    __shared__ __attribute__((aligned(16))) T ws[2][FX_KC][FX_WLD];   // W chunk [k][n]
    __shared__ __attribute__((aligned(16))) T xs[2][FX_MB][FX_LD];    // X chunk [row][k]
    __shared__ int kidx[LSTM_SD_MAX_K];
    if ((int)blockIdx.y >= a.T) {              // the transposes riding on this launch
        const long lin = ((long)(blockIdx.y - a.T) * gridDim.z + blockIdx.z) * gridDim.x + blockIdx.x;
        if (lin < (long)a.tr_gx * a.tr_gy * a.tr_gz) {
            const int bx = (int)(lin % a.tr_gx), by = (int)(lin / a.tr_gx % a.tr_gy), bz = (int)(lin / ((long)a.tr_gx * a.tr_gy));
            transpose_block<T>(a.tr, a.trN, bx, by, bz, a.tr_gx, a.tr_gy, (T(*)[33])&xs[0][0][0]);
        }
        return;
    }
    const int ctile = xcd_tile(blockIdx.x, (a.G + FX_NB - 1) / FX_NB);
    if (ctile < 0) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int t = blockIdx.y, m0 = blockIdx.z * FX_MB, n0 = ctile * FX_NB;
    const int g8 = 8 * (lane >> 4), cl = lane & 15;
    const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
    const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
    const int cnt = a.site.count[t];
    for (int j = tid; j < cnt; j += blockDim.x) {
        const int k = krow[j];
        kidx[j] = (DENSE && !mrow[j]) ? -1 : k;        // dense mode: the keep list is the identity
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t wr = buf_rsrc(a.W, (uint32_t)a.K * a.G * ES);
    const T* X = (const T*)a.X + (size_t)t * a.B * a.ldx;

    // staging roles: W row r = tid/8, 16 columns at 16*(tid%8); X row tid/8, 4 kept columns at 4*(tid%8)
    const int sr = tid >> 3, sq = tid & 7;
    constexpr int WNW = 16 * (int)ES / 16;             // 16-byte loads per W segment (2 bf16, 4 f32)
    u32x4_t wreg[WNW];
    T xreg[4];
    auto fetch = [&](int kc) {
        const int j = kc + sr;
        const int k = j < cnt ? kidx[j] : -1;
        const uint32_t off = ((uint32_t)max(k, 0) * a.G + n0 + 16 * sq) * ES;
#pragma unroll
        for (int q = 0; q < WNW; ++q) wreg[q] = __builtin_amdgcn_raw_buffer_load_b128(wr, off + 16 * q, 0, 0);
        const int row = m0 + sr;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int jj = kc + 4 * sq + q;
            const int kk = jj < cnt ? kidx[jj] : -1;
            xreg[q] = (kk >= 0 && row < a.B) ? X[(size_t)row * a.ldx + kk] : zero_val<T>();
        }
    };
    auto commit = [&](int buf) {
        uint4* wd = (uint4*)&ws[buf][sr][16 * sq];
#pragma unroll
        for (int q = 0; q < WNW; ++q) wd[q] = make_uint4(wreg[q][0], wreg[q][1], wreg[q][2], wreg[q][3]);
#pragma unroll
        for (int q = 0; q < 4; ++q) xs[buf][sr][4 * sq + q] = xreg[q];
    };

    f32x4_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[i][c] = f32x4_t{0, 0, 0, 0};
    const int nchunk = (cnt + FX_KC - 1) / FX_KC;
    if (nchunk > 0) {
        fetch(0);
        commit(0);
    }
    __syncthreads();
    for (int ch = 0; ch < nchunk; ++ch) {
        const int buf = ch & 1;
        if (ch + 1 < nchunk) fetch((ch + 1) * FX_KC);
        if constexpr (sizeof(T) == 2) {
            // A: 8 consecutive kept columns of the lane's row, one 16-byte
            // read; B: column n of the K-major W chunk over 8 rows, two
            // transposing reads (lanes 4e..4e+3 of a 16-lane group address
            // columns 0, 4, 8, 12 of row e; lane i receives column i)
            Raw8<T> fa[2], fb[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) raw_lds(fa[i], &xs[buf][16 * i + cl][g8]);
            const int e4 = (lane & 15) >> 2, j4 = lane & 3;
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                const int nb = 32 * w + 16 * c + 4 * j4;
                const uint2 lo = lds_tr4(&ws[buf][g8 + e4][nb]), hi = lds_tr4(&ws[buf][g8 + 4 + e4][nb]);
                fb[c].w[0] = lo.x; fb[c].w[1] = lo.y; fb[c].w[2] = hi.x; fb[c].w[3] = hi.y;
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int c = 0; c < 2; ++c) raw_mma(fa[i], fb[c], acc[i][c]);
        } else {
            Frag<T> fa[2], fb[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int e = 0; e < 8; ++e) fa[i].v[e] = xs[buf][16 * i + cl][g8 + e];
#pragma unroll
            for (int c = 0; c < 2; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) fb[c].v[e] = ws[buf][g8 + e][32 * w + 16 * c + cl];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int c = 0; c < 2; ++c) mma_16x16x32(fa[i], fb[c], acc[i][c]);
        }
        if (ch + 1 < nchunk) commit(buf ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int n = n0 + 32 * w + 16 * c + cl;
        if (n >= a.G) continue;
        const float bn = a.bias[n];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + 16 * i + acc_row(lane, r);
                if (row < a.B) a.Gx[((size_t)t * a.B + row) * a.G + n] = a.s * acc[i][c][r] + bn;
            }
    }
}

// ---------------------------------------------------------------------------
// One recurrent forward step (Eq. 1-6) fused with the gate pointwise.
// grid (ceil(H/(4NT)), ceil(B/(64/NT)), D), block 1024 (16 waves).  A
// workgroup owns 4*NT hidden units, i.e. NT 16-column tiles holding the
// four gates of 4 units each, for 64/NT batch rows; the contraction over
// the kept recurrent neurons is split over the 16 waves and reduced in LDS.
template <typename T, int NT>
__global__ void __launch_bounds__(1024) k_step(StepArgs a) {
    constexpr int MG = 64 / NT, MT = MG / 16, UPW = 4 * NT;
    __shared__ int kidx[LSTM_SD_MAX_K];
    __shared__ float red[16][MG][16 * NT + 1];
    const StepDir& D = a.d[blockIdx.z];
    const int utile = xcd_tile(blockIdx.x, (a.H + UPW - 1) / UPW);
    if (utile < 0) return;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int H = a.H, G = 4 * H, B = a.B;
    const int u0 = utile * UPW;
    const int m0 = blockIdx.y * MG;
    const int g8 = 8 * (lane >> 4);
    const T* hp = (const T*)D.hprev;
    const T* U = (const T*)D.U;
    const int cnt = *D.count;
    for (int j = threadIdx.x; j < cnt; j += blockDim.x) {
        const int k = D.keep[j];
        kidx[j] = (a.dense && !D.mask[k]) ? -1 : k;
    }
    __syncthreads();
    int gcol[NT];
    bool cok[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int c = lane & 15;
        const int unit = u0 + 4 * nt + (c & 3);
        cok[nt] = unit < H;
        gcol[nt] = (c >> 2) * H + unit;
    }
    f32x4_t acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
    for (int kc = 32 * w; kc < cnt; kc += 32 * 16) {
        int kk[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int j = kc + g8 + e;
            kk[e] = j < cnt ? kidx[j] : -1;
        }
        Frag<T> fb[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                fb[nt].v[e] = (kk[e] >= 0 && cok[nt]) ? U[(size_t)kk[e] * G + gcol[nt]] : zero_val<T>();
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int row = m0 + mt * 16 + (lane & 15);
            const bool rok = row < B;
            Frag<T> fa;
#pragma unroll
            for (int e = 0; e < 8; ++e) fa.v[e] = (kk[e] >= 0 && rok) ? hp[(size_t)row * H + kk[e]] : zero_val<T>();
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) mma_16x16x32(fa, fb[nt], acc[mt][nt]);
        }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[w][mt * 16 + acc_row(lane, r)][nt * 16 + (lane & 15)] = acc[mt][nt][r];
    __syncthreads();
    if (threadIdx.x < MG * UPW) {
        const int rr = threadIdx.x / UPW, uu = threadIdx.x % UPW;
        const int b = m0 + rr, u = u0 + uu;
        if (b < B && u < H) {
            const int nt = uu >> 2, cu = uu & 3;
            float pre[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int cc = nt * 16 + g * 4 + cu;
                float v = 0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) v += red[i][rr][cc];
                pre[g] = a.s * v + D.gx[(size_t)b * G + g * H + u];
            }
            const float ig = sigmoid_fast(pre[0]);
            const float fg = sigmoid_fast(pre[1]);
            const float gg = tanh_fast(pre[2]);
            const float og = sigmoid_fast(pre[3]);
            const float cp = D.cT[(size_t)b * H + u];
            const float cn = fg * cp + ig * gg;
            const float hn = og * tanh_fast(cn);
            const bool valid = (a.lengths == nullptr) || (D.t < a.lengths[b]);
            *(float4*)(D.gates + (size_t)b * G + 4 * u) = make_float4(ig, fg, gg, og);
            D.cres[(size_t)b * H + u] = valid ? cn : cp;
            const T hv = valid ? from_f32<T>(hn) : hp[(size_t)b * H + u];
            ((T*)D.hrec)[(size_t)b * H + u] = hv;
            ((T*)D.hrecT)[(size_t)u * a.BP + b] = hv;
            if (valid) {
                D.cT[(size_t)b * H + u] = cn;
                D.hT[(size_t)b * H + u] = hn;
            }
            if (D.y) D.y[(size_t)b * a.ldy + u] = valid ? hn : 0.0f;
            if (D.ybuf) {
                const T yv = valid ? from_f32<T>(hn) : zero_val<T>();
                ((T*)D.ybuf)[(size_t)b * a.ldy + u] = yv;
                ((T*)D.ybufT)[(size_t)u * a.BP + b] = yv;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// One BPTT step (per direction, grid.z).  grid (nkt + ceil(H/16),
// ceil(B/64), D), block 1024 (16 waves).
//   * workgroups x < nkt own 16 units kept at the previously processed step:
//     they first form the output-sparse recurrent gradient of those units,
//     dh_rec[b][u] = s * m * sum_n DA_next[b][n] U[u][n] (Eq. 10), with the
//     contraction over 4H split across the 16 waves;
//   * the other workgroups own 16 units dropped at that step (no product).
// Every workgroup then runs the pointwise backward of its units at t.  In
// the final pass (after the last step) it writes dh0 and dc0 instead.
template <typename T>
__global__ void __launch_bounds__(1024) k_bwd(BwdArgs a) {
    __shared__ float red[16][64][17];
    __shared__ int units[16];
    const BwdDir& D = a.d[blockIdx.z];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int H = a.H, G = 4 * H, B = a.B;
    const int m0 = blockIdx.y * 64;
    // Slot -> (XCD slice x, tile i of that slice).  Slice x holds units
    // [floor(xH/8), floor((x+1)H/8)), so a unit is always handled on the same
    // XCD and its rows of U stay in that XCD's L2 from step to step.
    const int nkslots = a.has_next ? NXCD * a.tps : 0;
    const bool kept_tile = (int)blockIdx.x < nkslots;
    const int slot = kept_tile ? blockIdx.x : blockIdx.x - nkslots;
    const int x = slot % NXCD, ti = slot / NXCD;
    int lo, hi;
    const int32_t* list;
    if (kept_tile) {
        lo = D.nkseg[2 * x]; hi = D.nkseg[2 * x + 2]; list = D.nkeep;
    } else if (a.has_next) {
        lo = D.ndseg[2 * x]; hi = D.ndseg[2 * x + 2]; list = D.ndrop;
    } else {
        lo = slice_start(x, H); hi = slice_start(x + 1, H); list = nullptr;
    }
    const int j0 = lo + 16 * ti;
    if (ti >= a.tps || j0 >= hi) return;
    if (threadIdx.x < 16) {
        const int j = j0 + threadIdx.x;
        units[threadIdx.x] = j < hi ? (list ? list[j] : j) : -1;
    }
    __syncthreads();
    if (kept_tile) {
        const int ul = units[lane & 15];
        const int g8 = 8 * (lane >> 4);
        const T* DA = (const T*)D.da_next;
        const T* U = (const T*)D.U;
        f32x4_t acc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0, 0, 0, 0};
        const int mtiles = min(4, (B - m0 + 15) / 16);
        for (int nc = 32 * w; nc < G; nc += 32 * 16) {
            Frag<T> fb;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int n = nc + g8 + 4 * h;
                if (ul >= 0 && n < G) ld4(U + (size_t)ul * G + n, fb.v + 4 * h);
                else zero4(fb.v + 4 * h);
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                if (mt < mtiles) {
                    const int row = m0 + mt * 16 + (lane & 15);
                    Frag<T> fa;
                    // fragment-major DA: entries past B or 4H are never written
                    ld4(DA + frag_lane_off(nc >> 5, (m0 >> 4) + mt, lane, a.mtiles), fa.v);
                    ld4(DA + frag_lane_off(nc >> 5, (m0 >> 4) + mt, lane, a.mtiles) + 4, fa.v + 4);
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (row >= B || nc + g8 + e >= G) fa.v[e] = zero_val<T>();
                    mma_16x16x32(fa, fb, acc[mt]);
                }
            }
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[w][mt * 16 + acc_row(lane, r)][lane & 15] = acc[mt][r];
    }
    __syncthreads();
    // pointwise: thread -> (row rr, unit slot i)
    const int rr = threadIdx.x >> 4, i = threadIdx.x & 15;
    const int b = m0 + rr;
    const int u = units[i];
    float da4[4] = {0.f, 0.f, 0.f, 0.f};
    if (b < B && u >= 0) {
        float dh = D.dhc[(size_t)b * H + u];
        if (kept_tile) {
            float v = 0.f;
#pragma unroll
            for (int q = 0; q < 16; ++q) v += red[q][rr][i];
            const float sc = (a.dense && !D.nmask[u]) ? 0.0f : a.s;
            dh += sc * v;
        }
        if (a.final_pass) {
            D.dh0[(size_t)b * H + u] = dh;
            D.dc0[(size_t)b * H + u] = D.dcs[(size_t)b * H + u];
        } else {
            const bool valid = (a.lengths == nullptr) || (D.t < a.lengths[b]);
            if (valid) {
                if (D.dy) dh += D.dy[(size_t)b * a.ldy + u];
                if (D.dxc) {
                    const int p = D.dxpos[u];
                    if (p >= 0) dh += D.dxc[(size_t)b * a.lddx + p];
                }
            }
            const float dcin = D.dcs[(size_t)b * H + u];
            if (valid) {
                const float4 gt = *(const float4*)(D.gates + (size_t)b * G + 4 * u);
                const float ig = gt.x, fg = gt.y, gg = gt.z, og = gt.w;
                const float ct = D.cres[(size_t)b * H + u];
                const float cp = D.cprev[(size_t)b * H + u];
                const float tc = tanh_fast(ct);
                const float dout = dh * tc;                            // Eq. 7
                const float dc = dh * og * (1.0f - tc * tc) + dcin;    // Eq. 7
                da4[0] = dc * gg * ig * (1.0f - ig);                   // Eq. 9, sigmoid'
                da4[1] = dc * cp * fg * (1.0f - fg);                   // Eq. 8, sigmoid'
                da4[2] = dc * ig * (1.0f - gg * gg);                   // Eq. 9, tanh'
                da4[3] = dout * og * (1.0f - og);                      // Eq. 7, sigmoid'
                D.dcs[(size_t)b * H + u] = dc * fg;                    // Eq. 8
                D.dhc[(size_t)b * H + u] = 0.0f;
            } else {
                D.dhc[(size_t)b * H + u] = dh;                         // frozen row: pass through
            }
            T* dat = (T*)D.daT;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const T v = from_f32<T>(da4[g]);
                ((T*)D.da)[frag_off(b, g * H + u, a.mtiles)] = v;
                dat[(size_t)(g * H + u) * a.BP + b] = v;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Output-sparse input gradient, all t (Eq. 10), summed over directions.
// grid (32 * tps * ceil(T/4), 1, ceil(B/64)), block 256: 16 kept columns per
// workgroup, the contraction over 4H split over the 4 waves.  Workgroup i
// runs on XCD c = i % 8, which takes the steps t = c/2 (mod 4) and the W
// slices 4(c%2) .. 4(c%2)+3: a step's DA is read by 2 XCDs and a slice of W
// by 4 (DA of all steps and W are of about the same size).  With scatter,
// the output is the full-width gradient: kept columns go to their own
// positions, and the workgroup of (slice, tile) also writes the zeros of
// the same tile of the slice's dropped columns.
template <typename T, int MT>
__global__ void __launch_bounds__(256) k_dx(DxArgs a) {
    constexpr int U = sizeof(T) == 2 ? 4 : 2;           // 32-column chunks per wave loaded together
    constexpr uint32_t ES = sizeof(T);
    __shared__ float red[4][64][17];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // slot -> (step t, slice x, tile ti): kept rows of t inside slice x of W
    const int c = blockIdx.x % NXCD, jw = blockIdx.x / NXCD;
    const int t = (c >> 1) + 4 * (jw / (4 * a.tps));
    const int x = 4 * (c & 1) + (jw / a.tps) % 4, ti = jw % a.tps;
    if (t >= a.T) return;
    const int32_t* ks = a.site.kseg + (size_t)t * (NSEG + 1);
    const int hi = ks[2 * x + 2];
    const int j0 = ks[2 * x] + 16 * ti;
    const int m0 = blockIdx.z * 64;
    // a step whose recurrence timed out gets NaN in every output
    const bool failed = a.status && *a.status != 0;
    if (a.scatter && ti < a.tps) {
        const int32_t* ds = a.site.dseg + (size_t)t * (NSEG + 1);
        const int dj = ds[2 * x] + 16 * ti + (threadIdx.x & 15);
        if (dj < ds[2 * x + 2]) {
            const int kd = a.site.drop[(size_t)t * a.site.kmax + dj];
            for (int r = threadIdx.x >> 4; r < 16 * MT; r += 16)
                if (m0 + r < a.B) a.out[((size_t)t * a.B + m0 + r) * a.ldo + kd] = failed ? __builtin_nanf("") : 0.0f;
        }
    }
    if (ti >= a.tps || j0 >= hi) return;
    const int cnt = hi;                     // columns of this tile end at the slice end
    const int cl = lane & 15;
    const int j = j0 + cl;
    const int g8 = 8 * (lane >> 4);
    const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
    const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
    // absent columns (j past the slice) read row 0; their outputs are not stored
    const int kr = (j < cnt) ? krow[j] : 0;
    f32x4_t acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4_t{0, 0, 0, 0};
    for (int d = 0; d < a.D; ++d) {
        // DA_t is fragment-major; lanes of rows past B read 0 without moving
        // data
        const size_t das = (size_t)((a.G + 31) / 32) * a.mtiles * 512;
        const __amdgpu_buffer_rsrc_t dr = buf_rsrc((const T*)a.da[d] + (size_t)t * das, (uint32_t)(das * ES));
        const __amdgpu_buffer_rsrc_t wr = buf_rsrc(a.W[d], (uint32_t)a.K * a.G * ES);
        const uint32_t woff = ((uint32_t)kr * a.G + g8) * ES;
        for (int nc0 = 32 * w; nc0 < a.G; nc0 += 128 * U) {
            Raw8<T> fb[U], fa[U][MT];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t nc = nc0 + 128 * u;
                raw_load(fb[u], wr, woff + nc * ES);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    raw_load(fa[u][mt], dr, m0 + 16 * mt + cl < a.B ? (uint32_t)(frag_lane_off(nc >> 5, (m0 >> 4) + mt, lane, a.mtiles) * ES) : OOB_OFF);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int nc = nc0 + 128 * u;
                if (nc + 32 > a.G) {            // chunk reaches past G: zero the DA side there (never written)
                    uint32_t m[Raw8<T>::NW];
                    pad_mask<T>(nc + g8, a.G, m);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) raw_and(fa[u][mt], m);
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) raw_mma(fa[u][mt], fb[u], acc[mt]);
            }
        }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[w][mt * 16 + acc_row(lane, r)][cl] = acc[mt][r];
    __syncthreads();
    float* out = a.out + (size_t)t * a.B * a.ldo;
    for (int q = threadIdx.x; q < 16 * MT * 16; q += 256) {
        const int rr = q >> 4, c = q & 15;
        const int row = m0 + rr, jj = j0 + c;
        if (row < a.B && jj < cnt) {
            const int kk = krow[jj];
            const float sc = (a.dense && !mrow[kk]) ? 0.0f : a.s;
            out[(size_t)row * a.ldo + (a.scatter ? kk : jj)] =
                failed ? __builtin_nanf("") : sc * (red[0][rr][c] + red[1][rr][c] + red[2][rr][c] + red[3][rr][c]);
        }
    }
}

// ---------------------------------------------------------------------------
// Row-sparse weight gradient (Eq. 11; Sec. 3.2 WG).  grid (64 *
// ceil(G/1024), 1, problems), block 512 (8 waves), dynamic LDS (rows of a
// slice + 1) * WG_LDC floats.  Workgroup (i, z) owns, for problem z, a
// neuron slice x, the rows [floor(xK/8), floor((x+1)K/8)), and the 128
// gradient columns of a block cb (wg_slot: the column blocks of an XCD share
// their DA^T through its L2), over every time step (no partial sums).
// At each t the kept rows of the slice (keep-list entries kseg[t][x] ..
// kseg[t][x+1]) are taken in 16-row tiles; wave w multiplies them with its
// 16 DA^T columns and adds each tile into its columns of the LDS
// accumulator.  Waves own disjoint columns, so they run without barriers
// until the final write; the gathered rows are shared through the cache.
//
// The kernel is built to issue few vector-ALU instructions per MFMA: the
// operands are fetched with buffer loads (32-bit offsets, out-of-range reads
// return 0) into packed registers, only the padded batch entries are zeroed
// (one AND per register), and the A rows of absent tile rows are not zeroed
// at all: their products land in a spare LDS row, which is never read back.
// The gather is a chain of two loads (keep-list entries, then the rows they
// name), so each wave runs it ahead: while t is multiplied, the A rows and
// DA^T fragments of t+1 are in flight, those of t+2 go out, and so do the
// keep-list entries of t+4.  The steps run in windows of 64, whose keep-list ranges sit in
// LDS.  All kept rows of a step are distinct, so the LDS sums read
// every row of the step first and then write them.  Rows never kept stay
// zero.  Every wave also sums its DA^T fragments: the bias gradient.
constexpr int WG_NB = 128;                 // gradient columns per workgroup
constexpr int WG_CT = 2;                   // 16-column tiles per wave (each A fragment feeds WG_CT products)
constexpr int WG_NWV = WG_NB / (16 * WG_CT); // waves per half workgroup
constexpr int WG_LDC = WG_NB + 4;          // LDS accumulator row pitch (floats)
template <typename T>
struct WgTiles { static constexpr int N = 6; };   // 16-row tiles in registers at once
template <>
struct WgTiles<float> { static constexpr int N = 4; };

// Whether the two halves of a row-sparse weight-gradient workgroup split the
// t-range (each then takes every kept row of the slice, into an accumulator
// of its own): when one round of tiles holds the whole slice
template <typename T>
__host__ __device__ inline bool wgrad_tsplit(int K) { return (K + NXCD - 1) / NXCD <= 16 * (WgTiles<T>::N / 2); }
// LDS bytes of the row-sparse weight gradient for a K-row weight
template <typename T>
inline size_t wgrad_lds_bytes(int K) {
    return (size_t)(wgrad_tsplit<T>(K) ? 2 : 1) * ((K + NXCD - 1) / NXCD + 1) * WG_LDC * sizeof(float);
}

// Layout of the staged row-sparse kernel's LDS: the accumulator rows of the
// largest slice (+ a spare row), two stage buffers (DA^T: 8 fragment tiles;
// the kept rows: up to wgs_tiles tiles; their accumulator row offsets), and
// the keep-list ranges of every step
__host__ __device__ inline int wgs_rows(int K) { return (K + NXCD - 1) / NXCD; }
__host__ __device__ inline int wgs_tiles(int K) { return (wgs_rows(K) + 15) / 16; }
__host__ __device__ inline int wgs_stage_bytes(int K) { return (8 + wgs_tiles(K)) * 1024 + 16 * wgs_tiles(K) * 4; }
inline size_t wgs_lds_bytes(int K, int T) {
    return (size_t)(wgs_rows(K) + 1) * WG_LDC * 4 + 2 * (size_t)wgs_stage_bytes(K) + (size_t)T * 8;
}
constexpr int WGS_MAX_ROWS = 128;          // a stage buffer row per thread piece: 512 / 4
constexpr size_t WGS_MAX_LDS = 80 * 1024;  // two workgroups per CU

// workgroup i -> (row slice x, column block cb).  Workgroup i runs on XCD
// i % 8, which takes the column blocks i % 8 + 8j with every row slice: one
// XCD's L2 then holds its columns' DA^T (4H x B per step, the larger operand)
// for all of the slices, and each XCD reads 1/8 of it.  The grid has
// 64 * ceil(column blocks / 8) workgroups; those past the last block return.
__device__ __forceinline__ void wg_slot(int& x, int& cb) {
    const int i = blockIdx.x, j = i / NXCD;
    x = j % NXCD;
    cb = i % NXCD + NXCD * (j / NXCD);
}

template <typename T, bool MULTI>
__device__ __forceinline__ void wgrad_gather(const WgArgs& a, float* acc_lds) {
    constexpr int MAXT = WgTiles<T>::N / 2;     // 16-row tiles of a round
    constexpr int NW = Raw8<T>::NW;
    constexpr uint32_t ES = sizeof(T);
    // acc_lds: [rows of the slice + 1][WG_LDC], one per half when the halves split the t-range
    int x, cb;
    wg_slot(x, cb);
    if (cb * WG_NB >= a.G) return;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // (wave-uniform)
    const int col = lane & 15, g8 = 8 * (lane >> 4);
    const int rh = w / WG_NWV;                   // this wave's half of the workgroup
    const int c0 = 16 * WG_CT * (w % WG_NWV);    // this wave's columns within the block: WG_CT tiles
    const int n0 = cb * WG_NB, n = n0 + c0 + col;   // (columns n + 16h)
    const int r0 = slice_start(x, a.K), r1 = slice_start(x + 1, a.K);
    const int nrow = r1 - r0;
    // the halves take the even and odd steps (each every kept row of the
    // slice), or the kept rows of the slice's two segments (each every step)
    const bool tsplit = wgrad_tsplit<T>(a.K);
    const int ts = tsplit ? 2 : 1;               // the stride of this wave's steps
    for (int i = lane + 64 * rh; i < (tsplit ? 2 : 1) * (nrow + 1) * 16 * WG_CT; i += 128)
        acc_lds[(i / (16 * WG_CT)) * WG_LDC + c0 + i % (16 * WG_CT)] = 0.0f;
    float* accr = acc_lds + (tsplit ? rh * (nrow + 1) * WG_LDC : 0);   // this half's accumulator
    // keep-list ranges of slice x at the steps t0 .. t1-1 of a window, in LDS
    // (a table in registers would make the compiler wait for all loads
    // wherever it is read)
    __shared__ int segtab[3][64];                // segments 2x, 2x+1 and their end
    int t0 = 0, t1 = 0;
    const int sb = tsplit ? 0 : rh, se = tsplit ? 2 : rh + 1;
    auto seg_b = [&](int t) { return __builtin_amdgcn_readfirstlane(segtab[sb][t - t0]); };
    auto seg_e = [&](int t) { return __builtin_amdgcn_readfirstlane(segtab[se][t - t0]); };
    uint32_t pm0[NW], pmb[WG_CT][NW];          // batch-pad masks of chunk 0 (A side; B side adds n < G)
    pad_mask<T>(g8, a.B, pm0);
    uint32_t boff[WG_CT];                      // DA^T fragment offsets of the column tiles
#pragma unroll
    for (int h = 0; h < WG_CT; ++h) {
#pragma unroll
        for (int q = 0; q < NW; ++q) pmb[h][q] = n + 16 * h < a.G ? pm0[q] : 0u;
        boff[h] = (uint32_t)(min(n + 16 * h, a.G - 1) * a.BP + g8) * ES;
    }
    const uint32_t abytes = (uint32_t)a.K * a.BP * ES, bbytes = (uint32_t)a.G * a.BP * ES;
    const int spare = nrow * WG_LDC;
    const bool dbw = a.db && x == 0 && (tsplit || rh == 0);   // this wave sums bias-gradient terms

    // keep-list entries of the A-fragment rows of tiles jt0 .. jt0+MAXT-1 at t
    auto rows_issue = [&](int t, int jt0, int* kv) {
        const int jb = seg_b(t), je = seg_e(t);
        const __amdgpu_buffer_rsrc_t kr = buf_rsrc(a.site.keep + (size_t)t * a.site.kmax, (uint32_t)a.site.kmax * 4);
#pragma unroll
        for (int i = 0; i < MAXT; ++i) {
            const int j = jb + (jt0 + i) * 16 + col;
            const int jc = j < je ? j : 0;
            kv[i] = (int)__builtin_amdgcn_raw_buffer_load_b32(kr, (uint32_t)jc * 4, 0, 0);
        }
    };
    // row of each tile's A-fragment lane; absent rows read row 0 and add
    // into the spare row
    auto rows_resolve = [&](int t, int jt0, const int* kv, int* kk, int* la) {
        const int jb = seg_b(t), je = seg_e(t);
#pragma unroll
        for (int i = 0; i < MAXT; ++i) {
            // bitwise selects: a branch here would let the compiler sink the
            // loads of kv into it
            const int j = jb + (jt0 + i) * 16 + col;
            const int okm = -(int)(j < je);
            kk[i] = kv[i] & okm;
            la[i] = (__mul24(kv[i] - r0, WG_LDC) & okm) | (spare & ~okm);
        }
    };
    auto act_rsrc = [&](int t) {
        const T* act = (a.actT_first && t == a.t_first) ? (const T*)a.actT_first
                                                        : (const T*)a.actT + (long)(t + a.shift) * a.tstride;
        return buf_rsrc(act, abytes);
    };
    auto dat_rsrc = [&](int t) { return buf_rsrc((const T*)a.daT + (size_t)t * a.G * a.BP, bbytes); };
    auto a_issue = [&](__amdgpu_buffer_rsrc_t ar, int bc, const int* kk, Raw8<T>* fa) {
#pragma unroll
        for (int i = 0; i < MAXT; ++i) raw_load(fa[i], ar, (__umul24((uint32_t)kk[i], (uint32_t)a.BP) + bc + g8) * ES);
    };
    float dbacc[WG_CT] = {};
    // multiply the tiles (chunk-0 fragments already loaded) with both column
    // tiles, finish the other batch chunks, and add the tiles into their LDS
    // rows.  Tiles past nt hold no kept row and are skipped (a wave-uniform
    // branch: their loads went out a step earlier, in another iteration,
    // so no load is moved into it).  The products
    // are taken transposed (DA^T fragment as the left operand): the output
    // column of a lane is then its own A-fragment row, and its four values
    // are four adjacent gradient columns, so each lane adds one 16-byte piece
    // of its own row.
    auto finish = [&](__amdgpu_buffer_rsrc_t ar, __amdgpu_buffer_rsrc_t br, const int* kk, const int* la, int nt,
                      Raw8<T>* fa, const Raw8<T>* fb0, bool first_round) {
        f32x4_t acc[MAXT][WG_CT];
#pragma unroll
        for (int i = 0; i < MAXT; ++i) {
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) acc[i][h] = f32x4_t{0, 0, 0, 0};
            if (i < nt) {
                raw_and(fa[i], pm0);
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) raw_mma(fb0[h], fa[i], acc[i][h]);
            }
        }
        for (int bc = 32; MULTI && bc < a.B; bc += 32) {
            Raw8<T> fb[WG_CT];
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) raw_load(fb[h], br, boff[h] + (uint32_t)bc * ES);
            a_issue(ar, bc, kk, fa);
            uint32_t pm[NW];
            pad_mask<T>(bc + g8, a.B, pm);
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) {
                raw_and(fb[h], pm);
                if (n + 16 * h >= a.G) raw_and(fb[h], pmb[h]);   // pmb is all zero past G
                if (first_round) db_add_raw(fb[h], dbacc[h]);
            }
#pragma unroll
            for (int i = 0; i < MAXT; ++i) {
                if (i < nt) {
                    raw_and(fa[i], pm);
#pragma unroll
                    for (int h = 0; h < WG_CT; ++h) raw_mma(fb[h], fa[i], acc[i][h]);
                }
            }
        }
        // output r of this lane is gradient column 4*(lane/16)+r of the
        // column tile, in the lane's own row
        const int cq = c0 + 4 * (lane >> 4);
        float4 old[MAXT][WG_CT];
#pragma unroll
        for (int i = 0; i < MAXT; ++i)
            if (i < nt)
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) old[i][h] = *(const float4*)(accr + la[i] + cq + 16 * h);
#pragma unroll
        for (int i = 0; i < MAXT; ++i)
            if (i < nt)
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) {
                    float4 v = old[i][h];
                    v.x += a.s * acc[i][h][0];
                    v.y += a.s * acc[i][h][1];
                    v.z += a.s * acc[i][h][2];
                    v.w += a.s * acc[i][h][3];
                    *(float4*)(accr + la[i] + cq + 16 * h) = v;
                }
    };

    for (t0 = 0; t0 < a.T; t0 += 64) {
        t1 = min(a.T, t0 + 64);
        __syncthreads();                       // the previous window's table is no longer read
        if (threadIdx.x < t1 - t0) {
            const int32_t* ks = a.site.kseg + (size_t)(t0 + threadIdx.x) * (NSEG + 1) + 2 * x;
            segtab[0][threadIdx.x] = ks[0];
            segtab[1][threadIdx.x] = ks[1];
            segtab[2][threadIdx.x] = ks[2];
        }
        __syncthreads();
        // ring slots alternating over the wave's steps (stride ts): the A
        // rows, DA^T fragments and LDS row addresses of its next two steps,
        // the keep-list entries of the two after
        int kv[2][MAXT], kk[2][MAXT], la[2][MAXT];
        Raw8<T> fa[2][MAXT], fb[2][WG_CT];
        // the operands of step t into slot sl, from its keep-list entries
        auto prime = [&](int t, int sl) {
            rows_resolve(t, 0, kv[sl], kk[sl], la[sl]);
            const __amdgpu_buffer_rsrc_t br = dat_rsrc(t);
            a_issue(act_rsrc(t), 0, kk[sl], fa[sl]);
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) raw_load(fb[sl][h], br, boff[h]);
        };
        // step t from slot sl (none past the window); then the slot takes
        // the operands of t+2ts and the keep-list entries of t+4ts.  Loads that
        // always go out (steps clamped into the window) and the same issue
        // order in the prologue keep the wait counts exact.
        auto step = [&](int t, int sl) {
            if (t < t1) {
                const __amdgpu_buffer_rsrc_t ar = act_rsrc(t), br = dat_rsrc(t);
                const int ntile = (seg_e(t) - seg_b(t) + 15) >> 4;
                Raw8<T> fb0[WG_CT];
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) {
                    fb0[h] = fb[sl][h];
                    raw_and(fb0[h], pmb[h]);
                    if (dbw) db_add_raw(fb0[h], dbacc[h]);
                }
                finish(ar, br, kk[sl], la[sl], min(ntile, MAXT), fa[sl], fb0, dbw);
                for (int jt0 = MAXT; MULTI && jt0 < ntile; jt0 += MAXT) {   // more kept rows than one round
                    int kv2[MAXT], kc[MAXT], lc[MAXT];
                    Raw8<T> fa2[MAXT];
                    rows_issue(t, jt0, kv2);
                    rows_resolve(t, jt0, kv2, kc, lc);
                    a_issue(ar, 0, kc, fa2);
                    finish(ar, br, kc, lc, min(ntile - jt0, MAXT), fa2, fb0, false);
                }
            }
            prime(min(t + 2 * ts, t1 - 1), sl);
            rows_issue(min(t + 4 * ts, t1 - 1), 0, kv[sl]);
        };
        const int tb = t0 + (tsplit ? rh : 0);
        rows_issue(min(tb, t1 - 1), 0, kv[0]);
        rows_issue(min(tb + ts, t1 - 1), 0, kv[1]);
        prime(min(tb, t1 - 1), 0);
        rows_issue(min(tb + 2 * ts, t1 - 1), 0, kv[0]);
        prime(min(tb + ts, t1 - 1), 1);
        rows_issue(min(tb + 3 * ts, t1 - 1), 0, kv[1]);
        for (int t = tb; t < t1; t += 2 * ts) {
            step(t, 0);
            step(t + ts, 1);
        }
    }
    __syncthreads();
    if (a.db && x == 0) {                      // lanes l, l+16, l+32, l+48 hold column l (+16)
        float v[WG_CT];
#pragma unroll
        for (int h = 0; h < WG_CT; ++h) {
            v[h] = dbacc[h];
            v[h] += __shfl_xor(v[h], 16);
            v[h] += __shfl_xor(v[h], 32);
        }
        // the odd half's sums pass through the (no longer used) spare row
        float* sp = acc_lds + nrow * WG_LDC + c0;
        if (tsplit && rh && lane < 16) {
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) sp[16 * h + lane] = v[h];
        }
        __syncthreads();
#pragma unroll
        for (int h = 0; h < WG_CT; ++h)
            if (!rh && lane < 16 && n + 16 * h < a.G) a.db[n + 16 * h] = tsplit ? v[h] + sp[16 * h + lane] : v[h];
    }
    float* out = a.out;
    const float* acc2 = acc_lds + (nrow + 1) * WG_LDC;   // the odd half's accumulator
    for (int i = threadIdx.x; i < nrow * WG_NB; i += blockDim.x) {
        const int rr = i / WG_NB, cc = i % WG_NB;
        if (n0 + cc < a.G)
            out[(size_t)(r0 + rr) * a.G + n0 + cc] =
                tsplit ? acc_lds[rr * WG_LDC + cc] + acc2[rr * WG_LDC + cc] : acc_lds[rr * WG_LDC + cc];
    }
}

// Row-sparse weight gradient with LDS-staged operands (bf16, batch <= 32,
// slices of at most 128 rows).  Same grid, slots and result as the kernel
// above; what differs is how a step's operands reach the waves.  There,
// every wave loaded its own fragments from memory: the four waves of a half
// the same gathered rows, the two halves the same DA^T columns, so the
// vector memory pipe moved about three times the step's data and set the
// step time.  Here the 512 threads load a step's operands once, one 16-byte
// piece each: a piece is 8 batch entries of a DA^T column of the block (8
// KB, one piece per thread) and of a kept row of the step in the slice
// (gathered through the keep list; absent rows read past the resource,
// i.e. zeros), and the threads store them fragment-major in LDS, with
// the accumulator row offset of each kept row beside them.  Wave w then
// multiplies DA^T column tile w with every kept-row tile of the step and
// adds the tiles into its 16 columns of the LDS accumulator.  Loads run two
// steps ahead of the store into LDS (register ring), keep-list entries two
// steps ahead of those; the stage buffers alternate, one barrier per step.
// The slice's keep-list ranges for every step sit in LDS ([T][2] ints).
template <typename T>
__device__ __forceinline__ void wgrad_staged(const WgArgs& a, float* lds) {
    static_assert(sizeof(T) == 2, "bf16 only");
    int x, cb;
    wg_slot(x, cb);
    if (cb * WG_NB >= a.G) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);     // (wave-uniform)
    const int n0 = cb * WG_NB;
    const int r0 = slice_start(x, a.K), nrow = slice_start(x + 1, a.K) - r0;
    const int ntmax = wgs_tiles(a.K);
    float* acc = lds;                                              // [rows of the slice + 1][WG_LDC]
    char* stg = (char*)(lds + (size_t)(wgs_rows(a.K) + 1) * WG_LDC);
    const int sbytes = wgs_stage_bytes(a.K);                       // one stage buffer
    int* seg = (int*)(stg + 2 * sbytes);                           // [T][2]: keep-list range of the slice
    for (int i = tid; i < (nrow + 1) * WG_NB; i += blockDim.x) acc[(i / WG_NB) * WG_LDC + i % WG_NB] = 0.0f;
    for (int t = tid; t < a.T; t += blockDim.x) {
        const int32_t* ks = a.site.kseg + (size_t)t * (NSEG + 1) + 2 * x;
        seg[2 * t] = ks[0];
        seg[2 * t + 1] = ks[2];
    }
    __syncthreads();

    // this thread's piece: row / column j of the step, batch entries 8q .. 8q+7
    // (lane l of a wave takes fragment position l of a 16-row tile: a wave's
    // LDS stores are one contiguous 1 KB block, free of bank conflicts)
    const int j = (tid & 15) + 16 * (tid >> 6), q = (tid >> 4) & 3;
    uint32_t pm[4];
    pad_mask<T>(8 * q, a.B, pm);
    const uint32_t abytes = (uint32_t)a.K * a.BP * 2, bbytes = (uint32_t)a.G * a.BP * 2;
    const uint32_t boff = n0 + j < a.G ? (uint32_t)((n0 + j) * a.BP + 8 * q) * 2 : OOB_OFF;
    const int frag = ((j & 15) + 16 * q) * 16 + (j >> 4) * 1024;   // fragment-major LDS offset of the piece
    const bool arow = j < 16 * ntmax;                              // a row of the stage buffer
    const int spare = nrow * WG_LDC;
    const uint32_t kbytes = (uint32_t)a.site.kmax * 4;
    auto clampt = [&](int t) { return t < a.T ? t : a.T - 1; };
    auto act_rsrc = [&](int t) {
        const T* act = (a.actT_first && t == a.t_first) ? (const T*)a.actT_first
                                                        : (const T*)a.actT + (long)(t + a.shift) * a.tstride;
        return buf_rsrc(act, abytes);
    };
    // ring slots: keep-list entry, staged pieces and accumulator row offset of a step
    int kv[2], la[2];
    uint4 ra[2], rb[2];
    auto issue_kv = [&](int t, int sl) {
        t = clampt(t);
        const int jb = seg[2 * t], n = seg[2 * t + 1] - jb;
        const __amdgpu_buffer_rsrc_t kr = buf_rsrc(a.site.keep + (size_t)t * a.site.kmax, kbytes);
        kv[sl] = (int)__builtin_amdgcn_raw_buffer_load_b32(kr, j < n ? (uint32_t)(jb + j) * 4 : OOB_OFF, 0, 0);
    };
    auto issue_ab = [&](int t, int sl) {
        t = clampt(t);
        const int n = seg[2 * t + 1] - seg[2 * t];
        const bool ok = j < n;
        const u32x4_t va = __builtin_amdgcn_raw_buffer_load_b128(
            act_rsrc(t), ok ? ((uint32_t)kv[sl] * a.BP + 8 * q) * 2 : OOB_OFF, 0, 0);
        const u32x4_t vb = __builtin_amdgcn_raw_buffer_load_b128(
            buf_rsrc((const T*)a.daT + (size_t)t * a.G * a.BP, bbytes), boff, 0, 0);
        ra[sl] = make_uint4(va[0], va[1], va[2], va[3]);
        rb[sl] = make_uint4(vb[0], vb[1], vb[2], vb[3]);
        la[sl] = ok ? (kv[sl] - r0) * WG_LDC : spare;
    };
    auto stage = [&](int buf, int sl) {
        char* sb = stg + buf * sbytes;
        const uint4 b4 = make_uint4(rb[sl].x & pm[0], rb[sl].y & pm[1], rb[sl].z & pm[2], rb[sl].w & pm[3]);
        *(uint4*)(sb + frag) = b4;
        if (arow) {
            const uint4 a4 = make_uint4(ra[sl].x & pm[0], ra[sl].y & pm[1], ra[sl].z & pm[2], ra[sl].w & pm[3]);
            *(uint4*)(sb + 8 * 1024 + frag) = a4;
            if (q == 0) ((int*)(sb + (8 + ntmax) * 1024))[j] = la[sl];
        }
    };
    const bool dbw = a.db && x == 0;
    float dbacc = 0.0f;
    const int cq = 16 * w + 4 * (lane >> 4);                       // this lane's 4 accumulator columns
    auto compute = [&](int t, int buf) {
        const char* sb = stg + buf * sbytes;
        const int n = __builtin_amdgcn_readfirstlane(seg[2 * t + 1] - seg[2 * t]);
        const int ntile = (n + 15) >> 4;
        Raw8<T> fb;
        raw_lds(fb, (const T*)(sb + w * 1024 + lane * 16));
        if (dbw) db_add_raw(fb, dbacc);
        const int* lab = (const int*)(sb + (8 + ntmax) * 1024);
        for (int rt0 = 0; rt0 < ntile; rt0 += 4) {
            Raw8<T> fa[4];
            int lr[4];
            f32x4_t d[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (rt0 + i < ntile) {
                    raw_lds(fa[i], (const T*)(sb + 8 * 1024 + (rt0 + i) * 1024 + lane * 16));
                    lr[i] = lab[(rt0 + i) * 16 + (lane & 15)];
                }
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (rt0 + i < ntile) {
                    d[i] = f32x4_t{0, 0, 0, 0};
                    raw_mma(fb, fa[i], d[i]);
                }
            float4 old[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (rt0 + i < ntile) old[i] = *(const float4*)(acc + lr[i] + cq);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (rt0 + i < ntile) {
                    float4 v = old[i];
                    v.x += a.s * d[i][0];
                    v.y += a.s * d[i][1];
                    v.z += a.s * d[i][2];
                    v.w += a.s * d[i][3];
                    *(float4*)(acc + lr[i] + cq) = v;
                }
        }
    };
    // step t: stage t+1 (its loads went out two steps earlier), issue the
    // operand loads of t+3 and the keep-list entries of t+5, multiply t
    auto iter = [&](int t, int sl) {
        stage((t + 1) & 1, sl ^ 1);
        issue_ab(t + 3, sl ^ 1);
        issue_kv(t + 5, sl ^ 1);
        if (t < a.T) compute(t, t & 1);
        __syncthreads();
    };
    issue_kv(0, 0);
    issue_kv(1, 1);
    issue_ab(0, 0);
    issue_kv(2, 0);
    issue_ab(1, 1);
    issue_kv(3, 1);
    stage(0, 0);
    issue_ab(2, 0);
    issue_kv(4, 0);
    __syncthreads();
    for (int t = 0; t < a.T; t += 2) {
        iter(t, 0);
        iter(t + 1, 1);
    }
    if (dbw) {                                                     // lanes l, l+16, l+32, l+48 hold column l
        dbacc += __shfl_xor(dbacc, 16);
        dbacc += __shfl_xor(dbacc, 32);
        if (lane < 16 && n0 + 16 * w + lane < a.G) a.db[n0 + 16 * w + lane] = dbacc;
    }
    for (int i = tid; i < nrow * WG_NB; i += blockDim.x) {
        const int rr = i / WG_NB, cc = i % WG_NB;
        if (n0 + cc < a.G) a.out[(size_t)(r0 + rr) * a.G + n0 + cc] = acc[rr * WG_LDC + cc];
    }
}

// Weight gradient of a full problem (identity keep lists, the dense
// comparison mode, or a row-sparse problem routed here: in the last two the
// mask byte zeroes the dropped rows) with LDS-staged rows (bf16, batch <=
// 32).  Same grid and slots as the kernels above.
// Wave w owns CT DA^T column tiles of the block (16 columns each, their
// fragments loaded straight into registers: no other wave reads them) and
// every row of the slice, in passes of up to 6 row tiles whose accumulators
// stay in registers over all steps.  The rows are the operand every wave
// shares: the workgroup loads a step's rows once (16-byte pieces: 8 batch
// entries of one row, zeroed when the row is dropped) and stores them
// fragment-major in LDS, where each wave reads its fragments; each fragment
// read feeds CT products.  Loads run three steps ahead (register ring), the
// two stage buffers alternate, one barrier per step.  8/CT waves.
constexpr int WFS_TILES = 6;               // 16-row tiles of a pass
constexpr int WFS_RING = 3;                // steps whose loads are in flight
constexpr size_t WFS_LDS = 2 * WFS_TILES * 1024;

template <typename T, bool MASKED, int CT = 1>
__device__ __forceinline__ void wgrad_full_staged(const WgArgs& a, float* lds) {
    static_assert(sizeof(T) == 2, "bf16 only");
    constexpr int NTH = 512 / CT;                               // threads
    constexpr int PP = (64 * WFS_TILES + NTH - 1) / NTH;        // staged pieces per thread and step
    int x, cb;
    wg_slot(x, cb);
    if (cb * WG_NB >= a.G) return;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);     // (wave-uniform)
    const int n0 = cb * WG_NB, g8 = 8 * (lane >> 4);
    int nc[CT];
#pragma unroll
    for (int h = 0; h < CT; ++h) nc[h] = n0 + 16 * (CT * w + h) + (lane & 15);
    const int r0 = slice_start(x, a.K), r1 = slice_start(x + 1, a.K);
    char* stg = (char*)lds;
    // staging: piece i = tid + NTH*p is row j of the pass, 8-entry part q
    // (lane l of a wave takes fragment position l of a 16-row tile: its LDS
    // stores are free of bank conflicts)
    int sj[PP], sfrag[PP];
    uint32_t pm[PP][4];
#pragma unroll
    for (int p = 0; p < PP; ++p) {
        const int i = tid + NTH * p, j = (i & 15) + 16 * (i >> 6), q = (i >> 4) & 3;
        sj[p] = j < 16 * WFS_TILES ? j : -1;
        sfrag[p] = ((j & 15) + 16 * q) * 16 + (j >> 4) * 1024;   // fragment-major LDS offset of the piece
        pad_mask<T>(8 * q, a.B, pm[p]);
    }
    uint32_t pmb[CT][4], boff[CT];
#pragma unroll
    for (int h = 0; h < CT; ++h) {
        pad_mask<T>(g8, a.B, pmb[h]);
        if (nc[h] >= a.G) pmb[h][0] = pmb[h][1] = pmb[h][2] = pmb[h][3] = 0u;
        boff[h] = g8 < a.B ? (uint32_t)(min(nc[h], a.G - 1) * a.BP + g8) * 2 : OOB_OFF;   // (as the row pieces)
    }
    const uint32_t abytes = (uint32_t)a.K * a.BP * 2, bbytes = (uint32_t)a.G * a.BP * 2;
    const bool dbw = a.db && x == NXCD - 1;                        // (the last slice is never empty)
    const bool masked = MASKED || a.fullmask;                      // dropped rows zeroed by the mask byte
    // the bias gradient (the last slice's workgroups): each DA^T fragment
    // times a fragment of ones, i.e. its column sums, on the matrix cores
    f32x4_t dbacc[CT];
#pragma unroll
    for (int h = 0; h < CT; ++h) dbacc[h] = f32x4_t{0, 0, 0, 0};
    Raw8<T> ones;
#pragma unroll
    for (int q = 0; q < Raw8<T>::NW; ++q) ones.w[q] = 0x3f803f80u;       // bf16 1.0, twice
    auto act_rsrc = [&](int t) {
        const T* act = (a.actT_first && t == a.t_first) ? (const T*)a.actT_first
                                                        : (const T*)a.actT + (long)(t + a.shift) * a.tstride;
        return buf_rsrc(act, abytes);
    };
    for (int rp = r0; rp < r1; rp += 16 * WFS_TILES) {            // passes over the slice's rows
        const int nt = min(WFS_TILES, (r1 - rp + 15) >> 4);        // row tiles of the pass
        const bool first = rp == r0 && dbw;                        // (the bias gradient: first pass)
        bool rok[PP];
#pragma unroll
        for (int p = 0; p < PP; ++p) rok[p] = sj[p] >= 0 && rp + sj[p] < r1;
        // pieces wholly past the batch (entries 24-31 at B <= 24) read 0
        // without moving data, like rows past the slice
        bool aok[PP];
#pragma unroll
        for (int p = 0; p < PP; ++p) aok[p] = rok[p] && 8 * (((tid + NTH * p) >> 4) & 3) < a.B;
        uint4 ra[WFS_RING][PP];
        Raw8<T> rb[WFS_RING][CT];
        int mk[WFS_RING][PP];
        auto issue = [&](int t, int sl) {
            t = t < a.T ? t : a.T - 1;
            const __amdgpu_buffer_rsrc_t ar = act_rsrc(t);
            // (the mask load is always issued, past the resource when
            // unmasked: a load under a branch would make the compiler wait
            // for every load on its own)
            const __amdgpu_buffer_rsrc_t mr = buf_rsrc(a.site.mask + (size_t)t * a.site.kmax, (uint32_t)a.site.kmax);
#pragma unroll
            for (int p = 0; p < PP; ++p) {
                const int row = rp + sj[p], q = ((tid + NTH * p) >> 4) & 3;
                const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(
                    ar, aok[p] ? (uint32_t)(row * a.BP + 8 * q) * 2 : OOB_OFF, 0, 0);
                ra[sl][p] = make_uint4(v[0], v[1], v[2], v[3]);
                mk[sl][p] = (int)__builtin_amdgcn_raw_buffer_load_b8(mr, masked && rok[p] ? (uint32_t)row : OOB_OFF, 0, 0);
            }
            const __amdgpu_buffer_rsrc_t br = buf_rsrc((const T*)a.daT + (size_t)t * a.G * a.BP, bbytes);
#pragma unroll
            for (int h = 0; h < CT; ++h) raw_load(rb[sl][h], br, boff[h]);
        };
        auto stage = [&](int buf, int sl) {
#pragma unroll
            for (int p = 0; p < PP; ++p)
                if (sj[p] >= 0) {
                    uint4 v = make_uint4(ra[sl][p].x & pm[p][0], ra[sl][p].y & pm[p][1], ra[sl][p].z & pm[p][2],
                                         ra[sl][p].w & pm[p][3]);
                    if (masked && !mk[sl][p]) v = make_uint4(0u, 0u, 0u, 0u);
                    *(uint4*)(stg + buf * (WFS_TILES * 1024) + sfrag[p]) = v;
                }
        };
        f32x4_t acc[WFS_TILES][CT];
#pragma unroll
        for (int i = 0; i < WFS_TILES; ++i)
#pragma unroll
            for (int h = 0; h < CT; ++h) acc[i][h] = f32x4_t{0, 0, 0, 0};
        auto compute = [&](int buf, int sl) {
            Raw8<T> fb[CT];
#pragma unroll
            for (int h = 0; h < CT; ++h) {
                fb[h] = rb[sl][h];
                raw_and(fb[h], pmb[h]);
                if (first) raw_mma(fb[h], ones, dbacc[h]);
            }
            const char* sb = stg + buf * (WFS_TILES * 1024);
            // every tile, also past nt (their accumulators are never written
            // out): the LDS reads then go out together instead of one read,
            // wait and product at a time behind a branch
            Raw8<T> fa[WFS_TILES];
#pragma unroll
            for (int i = 0; i < WFS_TILES; ++i) raw_lds(fa[i], (const T*)(sb + i * 1024 + lane * 16));
#pragma unroll
            for (int i = 0; i < WFS_TILES; ++i)
#pragma unroll
                for (int h = 0; h < CT; ++h) raw_mma(fb[h], fa[i], acc[i][h]);
        };
        // step t: stage t+1 (its loads went out two steps earlier), multiply
        // t, then its slot takes the loads of t+3
        auto iter = [&](int t, int sl) {
            stage((t + 1) & 1, (sl + 1) % WFS_RING);
            if (t < a.T) compute(t & 1, sl);
            issue(t + WFS_RING, sl);
            __syncthreads();
        };
#pragma unroll
        for (int i = 0; i < WFS_RING; ++i) issue(i, i);
        stage(0, 0);
        __syncthreads();
        for (int t = 0; t < a.T; t += WFS_RING) {
#pragma unroll
            for (int i = 0; i < WFS_RING; ++i) iter(t + i, i);
        }
        // (transposed products) output r of this lane is gradient column
        // 4*(lane/16)+r of tile h, in the lane's own row
#pragma unroll
        for (int h = 0; h < CT; ++h) {
            const int nq = n0 + 16 * (CT * w + h) + 4 * (lane >> 4);
#pragma unroll
            for (int i = 0; i < WFS_TILES; ++i) {
                const int orow = rp + 16 * i + (lane & 15);
                if (i < nt && orow < r1) {
                    float* o = a.out + (size_t)orow * a.G + nq;
                    if (nq + 3 < a.G) {
                        *(float4*)o = make_float4(a.s * acc[i][h][0], a.s * acc[i][h][1], a.s * acc[i][h][2],
                                                  a.s * acc[i][h][3]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (nq + r < a.G) o[r] = a.s * acc[i][h][r];
                    }
                }
            }
        }
    }
    if (dbw && (lane & 15) == 0) {                                 // output r of lane 16j: column 4j+r's sum
#pragma unroll
        for (int h = 0; h < CT; ++h)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int n = n0 + 16 * (CT * w + h) + 4 * (lane >> 4) + r;
                if (n < a.G) a.db[n] = dbacc[h][r];
            }
    }
}

// Weight gradient of a site whose keep lists are all the identity (p = 0,
// or the dense comparison mode, where the mask zeroes the dropped rows):
// every row takes part at every t, so the accumulators stay in registers
// over the whole t-range; no gather, no scatter.  Same grid as the
// row-sparse kernel: workgroup i owns a slice x and 128 columns; wave
// w owns 32 columns (two tiles: each A fragment feeds two products) and
// the rows of the slice in passes of 16-row tiles.  The two halves of the
// workgroup (w / 4) split each pass's tiles, NTW each; a slice that one
// half's NTW tiles cover instead has the halves split the t-range (even and
// odd steps), each carrying half the serial chain, and add their sums
// through LDS at the end.  The operands of two of a wave's steps are in
// flight while one is multiplied.  The bias gradient comes from the workgroups of the
// last slice (never empty: it ends at K).
template <typename T, bool MASKED, int NTW, bool MULTI, int RING = 2>
__device__ __forceinline__ void wgrad_full(const WgArgs& a, float* red) {
    constexpr int NW = Raw8<T>::NW;
    constexpr uint32_t ES = sizeof(T);
    int x, cb;
    wg_slot(x, cb);
    if (cb * WG_NB >= a.G) return;
    const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // (wave-uniform)
    const int col = lane & 15, g8 = 8 * (lane >> 4);
    const int rh = w / WG_NWV;                 // this wave's half of the workgroup
    const int n = cb * WG_NB + 16 * WG_CT * (w % WG_NWV) + col;   // columns n + 16h
    const int r0 = slice_start(x, a.K), r1 = slice_start(x + 1, a.K);
    const bool tsplit = r1 - r0 <= 16 * NTW;   // the halves split the steps (else the tiles)
    const int t1 = a.T, tb = tsplit ? rh : 0, ts = tsplit ? 2 : 1;
    uint32_t pm0[NW], pmb[WG_CT][NW];          // batch-pad masks (B side also zero past G)
    pad_mask<T>(g8, a.B, pm0);
    uint32_t boff[WG_CT];
#pragma unroll
    for (int h = 0; h < WG_CT; ++h) {
#pragma unroll
        for (int q = 0; q < NW; ++q) pmb[h][q] = n + 16 * h < a.G ? pm0[q] : 0u;
        boff[h] = (uint32_t)(min(n + 16 * h, a.G - 1) * a.BP + g8) * ES;
    }
    const uint32_t abytes = (uint32_t)a.K * a.BP * ES, bbytes = (uint32_t)a.G * a.BP * ES;
    float dbacc[WG_CT] = {};
    const bool dbw = a.db && x == NXCD - 1;    // this workgroup sums the bias gradient
    auto act_rsrc = [&](int t) {
        const T* act = (a.actT_first && t == a.t_first) ? (const T*)a.actT_first
                                                        : (const T*)a.actT + (long)(t + a.shift) * a.tstride;
        return buf_rsrc(act, abytes);
    };
    auto dat_rsrc = [&](int t) { return buf_rsrc((const T*)a.daT + (size_t)t * a.G * a.BP, bbytes); };
    // this wave's slot of the pass reduction: [tile][half][reg][lane]
    float* mine = red + (w % WG_NWV) * (NTW * WG_CT * 4 * 64) + lane;

    for (int rp = r0; rp < r1; rp += 32 * NTW) {           // passes over the slice's row tiles
        const bool first = rp == r0 && dbw;    // (the bias gradient is summed on the first pass)
        const int rb = tsplit ? rp : rp + 16 * NTW * rh;   // this wave's first row of the pass
        int rowa[NTW];                         // A-fragment row of this lane in tile i (clamped into K)
#pragma unroll
        for (int i = 0; i < NTW; ++i) rowa[i] = min(rb + 16 * i + col, a.K - 1);
        f32x4_t acc[NTW][WG_CT];
#pragma unroll
        for (int i = 0; i < NTW; ++i)
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) acc[i][h] = f32x4_t{0, 0, 0, 0};
        // operands of two of the wave's steps in flight, slots alternating
        Raw8<T> fa[RING][NTW], fb[RING][WG_CT];
        int mk[RING][NTW];
        auto issue = [&](int t, int sl) {
            const __amdgpu_buffer_rsrc_t ar = act_rsrc(t), br = dat_rsrc(t);
#pragma unroll
            for (int i = 0; i < NTW; ++i) raw_load(fa[sl][i], ar, (uint32_t)(rowa[i] * a.BP + g8) * ES);
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) raw_load(fb[sl][h], br, boff[h]);
            if (MASKED) {
                const __amdgpu_buffer_rsrc_t mr = buf_rsrc(a.site.mask + (size_t)t * a.site.kmax, (uint32_t)a.site.kmax);
#pragma unroll
                for (int i = 0; i < NTW; ++i) mk[sl][i] = (int)__builtin_amdgcn_raw_buffer_load_b8(mr, (uint32_t)rowa[i], 0, 0);
            }
        };
        // the step in slot sl (none past the range); then that slot takes the
        // operands of step tn (loads that always go out keep the wait counts exact)
        auto step = [&](int t, int sl, int tn) {
          if (t < t1) {
            Raw8<T>(&ca)[NTW] = fa[sl];
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) {
                raw_and(fb[sl][h], pmb[h]);
                if (first) db_add_raw(fb[sl][h], dbacc[h]);
            }
#pragma unroll
            for (int i = 0; i < NTW; ++i) {
                raw_and(ca[i], pm0);
                if (MASKED) {
#pragma unroll
                    for (int q = 0; q < NW; ++q) ca[i].w[q] = mk[sl][i] ? ca[i].w[q] : 0u;
                }
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) raw_mma(fb[sl][h], ca[i], acc[i][h]);
            }
            for (int bc = 32; MULTI && bc < a.B; bc += 32) {    // further batch chunks (B > 32)
                const __amdgpu_buffer_rsrc_t ar = act_rsrc(t), br = dat_rsrc(t);
                Raw8<T> xb[WG_CT], xa[NTW];
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) raw_load(xb[h], br, boff[h] + (uint32_t)bc * ES);
#pragma unroll
                for (int i = 0; i < NTW; ++i) raw_load(xa[i], ar, (uint32_t)(rowa[i] * a.BP + bc + g8) * ES);
                uint32_t pm[NW];
                pad_mask<T>(bc + g8, a.B, pm);
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) {
                    raw_and(xb[h], pm);
                    if (n + 16 * h >= a.G) raw_and(xb[h], pmb[h]);   // pmb is all zero past G
                    if (first) db_add_raw(xb[h], dbacc[h]);
                }
#pragma unroll
                for (int i = 0; i < NTW; ++i) {
                    raw_and(xa[i], pm);
                    if (MASKED) {
#pragma unroll
                        for (int q = 0; q < NW; ++q) xa[i].w[q] = mk[sl][i] ? xa[i].w[q] : 0u;
                    }
#pragma unroll
                    for (int h = 0; h < WG_CT; ++h) raw_mma(xb[h], xa[i], acc[i][h]);
                }
            }
          }
            issue(tn, sl);
        };
        if (tb < t1) {
#pragma unroll
            for (int j = 0; j < RING; ++j) issue(min(tb + j * ts, t1 - 1), j);
        }
        for (int t = tb; t < t1; t += RING * ts) {
#pragma unroll
            for (int j = 0; j < RING; ++j) step(t + j * ts, j, min(t + (j + RING) * ts, t1 - 1));
        }
        // the odd half hands its sums to the even half
        if (tsplit && rh) {
#pragma unroll
            for (int i = 0; i < NTW; ++i)
#pragma unroll
                for (int h = 0; h < WG_CT; ++h)
#pragma unroll
                    for (int r = 0; r < 4; ++r) mine[((i * WG_CT + h) * 4 + r) * 64] = acc[i][h][r];
        }
        if (tsplit) __syncthreads();
        if (!tsplit || !rh) {
            // (transposed products) output r of this lane is gradient column
            // 4*(lane/16)+r of the column tile, in the lane's own row; G is a
            // multiple of 4, so the four columns are all in range or none
            const int nq = n - col + 4 * (lane >> 4);
#pragma unroll
            for (int i = 0; i < NTW; ++i) {
                const int row = rb + 16 * i + col;
#pragma unroll
                for (int h = 0; h < WG_CT; ++h) {
                    float4 v;
                    v.x = a.s * (tsplit ? acc[i][h][0] + mine[((i * WG_CT + h) * 4 + 0) * 64] : acc[i][h][0]);
                    v.y = a.s * (tsplit ? acc[i][h][1] + mine[((i * WG_CT + h) * 4 + 1) * 64] : acc[i][h][1]);
                    v.z = a.s * (tsplit ? acc[i][h][2] + mine[((i * WG_CT + h) * 4 + 2) * 64] : acc[i][h][2]);
                    v.w = a.s * (tsplit ? acc[i][h][3] + mine[((i * WG_CT + h) * 4 + 3) * 64] : acc[i][h][3]);
                    if (row < r1 && nq + 16 * h < a.G) *(float4*)(a.out + (size_t)row * a.G + nq + 16 * h) = v;
                }
            }
        }
        if (tsplit) __syncthreads();           // (the next pass reuses the slots)
    }
    if (dbw) {                                 // (the last slice is never empty) lanes l, l+16, l+32, l+48 hold column l
        if (tsplit && rh) {
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) mine[64 * h] = dbacc[h];
        }
        if (tsplit) __syncthreads();
        if (!rh) {
#pragma unroll
            for (int h = 0; h < WG_CT; ++h) {
                float v = tsplit ? dbacc[h] + mine[64 * h] : dbacc[h];
                v += __shfl_xor(v, 16);
                v += __shfl_xor(v, 32);
                if (lane < 16 && n + 16 * h < a.G) a.db[n + 16 * h] = v;
            }
        }
    }
}

// NaN into the part of a problem's outputs this workgroup owns (its row
// slice and column block; slice 0 also the bias)
__device__ __forceinline__ void wgrad_poison(const WgArgs& a) {
    int x, cb;
    wg_slot(x, cb);
    const int n0 = cb * WG_NB;
    const int r0 = slice_start(x, a.K), r1 = slice_start(x + 1, a.K);
    const float nan = __builtin_nanf("");
    for (int i = threadIdx.x; i < (r1 - r0) * WG_NB; i += blockDim.x) {
        const int rr = i / WG_NB, cc = i % WG_NB;
        if (n0 + cc < a.G) a.out[(size_t)(r0 + rr) * a.G + n0 + cc] = nan;
    }
    if (a.db && x == 0)
        for (int c = threadIdx.x; c < WG_NB; c += blockDim.x)
            if (n0 + c < a.G) a.db[n0 + c] = nan;
}

// LDS of the full kernel's pass reduction
template <typename T>
constexpr size_t wgrad_full_lds_bytes() { return (size_t)WG_NWV * (WgTiles<T>::N / 2) * WG_CT * 4 * 64 * 4; }

// One launch for every weight gradient of a pass (grid z = problem): a
// problem whose keep lists are all the identity takes the full kernel, the
// others the row-sparse one; either way every workgroup runs every step, so
// the two kinds overlap instead of taking a launch each.
template <typename T, bool MASKED, bool MULTI>
__global__ void __launch_bounds__(128 * WG_NWV) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 2 && !MULTI ? 4 : 1))) k_wgrad(WgBatch bt) {
    extern __shared__ float acc_lds[];
    const WgArgs& a = bt.p[blockIdx.z];
    if (bt.status && *bt.status != 0) {        // the step's recurrence timed out: NaN in every output
        wgrad_poison(a);
        return;
    }
    if (a.full) {
        if constexpr (sizeof(T) == 2) {
            if (a.staged) wgrad_full_staged<T, MASKED>(a, acc_lds);
            else wgrad_full<T, MASKED, WgTiles<T>::N / 2, MULTI>(a, acc_lds);
        } else wgrad_full<T, MASKED, WgTiles<T>::N / 2, MULTI>(a, acc_lds);
    } else if constexpr (sizeof(T) == 2) {
        if (a.staged) wgrad_staged<T>(a, acc_lds);
        else wgrad_gather<T, MULTI>(a, acc_lds);
    } else wgrad_gather<T, MULTI>(a, acc_lds);
}

// 4 waves of 2 column tiles: each row fragment read from LDS feeds two
// products (8 waves of one tile: 43 us at LM-medium against 41), 145
// registers, 3 waves per SIMD, 3 workgroups per CU
constexpr int WFS_FS_CT = 2;
constexpr int WFS_FS_THREADS = 512 / WFS_FS_CT;
constexpr int WFS_FS_WPE = 3;

// The same pass when every problem runs on the staged full kernel (bf16,
// batch <= 32): built on its own for three workgroups per CU, so that a
// pass's workgroups (the grid is 64 per 1024 gradient columns and problem)
// mostly run in one round.
template <bool MASKED>
__global__ void __launch_bounds__(WFS_FS_THREADS) __attribute__((amdgpu_waves_per_eu(WFS_FS_WPE))) k_wgrad_fs(WgBatch bt) {
    extern __shared__ float stage_lds[];
    const WgArgs& a = bt.p[blockIdx.z];
    if (bt.status && *bt.status != 0) {
        wgrad_poison(a);
        return;
    }
    wgrad_full_staged<bf16, MASKED, WFS_FS_CT>(a, stage_lds);
}

// ---------------------------------------------------------------------------
// Small elementwise kernels.

// the persistent kernels' barrier counters and error flag <- 0
__device__ __forceinline__ void clear_sync(unsigned* bar, int* err) {
    if (blockIdx.x == 0) {
        for (int i = threadIdx.x; i <= BAR_LINES * BAR_EXIT; i += blockDim.x) bar[BAR_PITCH * i] = 0u;
        if (threadIdx.x == 0) *err = 0;
    }
}


// carries <- dhT/dcT slices (or zero)
// and, when da is given, zero the columns 4H .. (last 32-column chunk end)
// of every fragment-major DA block (nblk blocks of das elements of es
// bytes): no kernel writes them, and the backward products read them
__global__ void k_bwd_init(const float* dhT, const float* dcT, float* dhc, float* dcs, long n,
                           void* da, int es, int G, int mtiles, long nblk, long das, unsigned* bar, int* err) {
    clear_sync(bar, err);
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        dhc[i] = dhT ? dhT[i] : 0.0f;
        dcs[i] = dcT ? dcT[i] : 0.0f;
    }
    const int padc = (G % 32) ? 32 - G % 32 : 0, rows = 16 * mtiles;
    const long np = da ? nblk * rows * padc : 0;
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < np; i += (long)gridDim.x * blockDim.x) {
        const long blk = i / (rows * padc), rem = i % (rows * padc);
        const size_t off = (size_t)blk * das + frag_off((int)(rem / padc), G + (int)(rem % padc), mtiles);
        if (es == 2) ((uint16_t*)da)[off] = 0;
        else ((uint32_t*)da)[off] = 0u;
    }
}

// Embedding-table gradient of a language model's input: the layer-0 input
// gradient dx_t[b] is added into row tokens[t][b] of d_emb, over the columns
// kept at t (the dropped columns of dx are zero, Eq. 10).  grid
// (ceil(V/EM_VB), ceil(I/EM_CW)): a workgroup owns EM_VB token ids and EM_CW
// columns (lane = column); block 256 (4 waves).  Wave w takes the position
// groups w, w+4, ... (64 positions each, ascending), loading the token ids of
// EM_TG groups at once, and lists the positions whose token it owns, in
// order, in LDS (a ballot and a prefix count per group).  It then walks its
// list EM_BATCH positions at a time (their dx values and mask bytes all in
// flight) and adds them into its own partial sums in LDS, in list order (a
// plain read-modify-write: LDS float atomics, back to back on the rows of a
// frequent token, were twice as slow), so each partial is summed in
// ascending position order.  Finally the wave that owns token j
// (j mod 4) adds the four partials in wave order and writes row j once (all
// its loads before its stores): a fixed summation order, no global atomics,
// the same result on every run.  A Zipf-distributed text puts most positions
// in the first workgroup's range; its four waves still share them.
constexpr int EM_VB = 64, EM_CW = 64, EM_BATCH = 16, EM_TG = 4, EM_LIST = 256;

__global__ void __launch_bounds__(256) k_emb_grad(const int32_t* tokens, int N, int B, int V, const float* dx,
                                                  SiteView nr0, int I, float* d_emb) {
    __shared__ float part[4][EM_VB][EM_CW];
    __shared__ int lpos[4][EM_LIST], lj[4][EM_LIST], lm[4][EM_LIST];   // position, token - v0, mask row offset
    __shared__ int touched[EM_VB];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int v0 = blockIdx.x * EM_VB;
    const int vn = min(EM_VB, V - v0);                 // token ids v0 .. v0+vn-1
    const int col = blockIdx.y * EM_CW + lane;
    const bool colok = col < I;
    const int colc = colok ? col : I - 1;              // lanes past I read a valid column, never written
    float4* pz = reinterpret_cast<float4*>(&part[w][0][0]);
    for (int i = lane; i < EM_VB * EM_CW / 4; i += 64) pz[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (tid < EM_VB) touched[tid] = 0;
    __syncthreads();
    // add the listed positions [0, nl) into this wave's partial sums
    auto drain = [&](int nl) {
        for (int k0 = 0; k0 < nl; k0 += EM_BATCH) {
            int sp[EM_BATCH], sj[EM_BATCH], sm[EM_BATCH];
#pragma unroll
            for (int k = 0; k < EM_BATCH; ++k) {
                const int e = min(k0 + k, nl - 1);     // (past the end: a listed position, not added)
                sp[k] = lpos[w][e];
                sj[k] = lj[w][e];
                sm[k] = lm[w][e];
            }
            float d[EM_BATCH];
            bool m[EM_BATCH];
#pragma unroll
            for (int k = 0; k < EM_BATCH; ++k) {
                d[k] = dx[(size_t)sp[k] * I + colc];
                m[k] = nr0.mask[(size_t)sm[k] + colc] != 0;
            }
#pragma unroll
            for (int k = 0; k < EM_BATCH; ++k)
                if (k0 + k < nl) part[w][sj[k]][lane] += m[k] ? d[k] : 0.0f;
            if (lane == 0)
                for (int k = 0; k < EM_BATCH && k0 + k < nl; ++k) touched[sj[k]] = 1;
        }
    };
    int nl = 0;                                        // (wave-uniform) listed positions
    for (int g0 = 64 * w; g0 < N; g0 += 256 * EM_TG) {
        int tk[EM_TG];
#pragma unroll
        for (int u = 0; u < EM_TG; ++u) {              // the token ids of EM_TG groups, loaded together
            const int pos = g0 + 256 * u + lane;
            tk[u] = pos < N ? tokens[pos] : -1;
        }
#pragma unroll
        for (int u = 0; u < EM_TG; ++u) {
            const int pos = g0 + 256 * u + lane;
            const bool act = tk[u] >= v0 && tk[u] - v0 < vn;   // (tk >= v0 >= 0: no wrap-around)
            const uint64_t bal = __builtin_amdgcn_ballot_w64(act);
            if (nl + 64 > EM_LIST) {                   // the list could overflow: drain it first
                drain(nl);
                nl = 0;
            }
            if (act) {
                const int r = __builtin_popcountll(bal & ((1ull << lane) - 1ull));
                lpos[w][nl + r] = pos;
                lj[w][nl + r] = tk[u] - v0;
                lm[w][nl + r] = (pos / B) * nr0.kmax;
            }
            nl += __builtin_popcountll(bal);
        }
    }
    drain(nl);
    __syncthreads();
    constexpr int NQ = EM_VB / 4;
    float tot[NQ], old[NQ];
    bool own[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int jj = w + 4 * q;
        own[q] = jj < vn && touched[jj] && colok;
        tot[q] = ((part[0][jj][lane] + part[1][jj][lane]) + part[2][jj][lane]) + part[3][jj][lane];
        old[q] = own[q] ? d_emb[(size_t)(v0 + jj) * I + col] : 0.0f;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q)
        if (own[q]) d_emb[(size_t)(v0 + w + 4 * q) * I + col] = old[q] + tot[q];
}

// ---------------------------------------------------------------------------
// Case-I dropout (the comparator of the paper's "NR+Random" baselines): one
// keep bit per element (t, b, k) of a layer input, drawn with the generator
// of the masks above with the batch row in the high word of the stream
// counter: counter (k/4, t, sid + 2^32 (b + 1), step), word k%4.
// dst = src * kept * s in the compute type; mask [T][B][K] bytes.
// grid (ceil(K/4 / 64), B, T), block 64: a thread draws 4 elements.
template <typename S, typename T>
__global__ void __launch_bounds__(64) k_case1_drop(const S* src, T* dst, uint8_t* mask, int B, int K, uint64_t seed,
                                                   uint64_t step, uint64_t sid, uint64_t thr, float s) {
    const int q = blockIdx.x * 64 + threadIdx.x, b = blockIdx.y, t = blockIdx.z;
    if (4 * q >= K) return;
    u64x4 c;
    c.x[0] = (uint64_t)q;
    c.x[1] = (uint64_t)t;
    c.x[2] = sid + ((uint64_t)(b + 1) << 32);
    c.x[3] = step;
    const u64x4 r = philox4x64_10(c, seed, 0ull);
    const size_t row = ((size_t)t * B + b) * K;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int k = 4 * q + e;
        if (k < K) {
            const uint8_t kept = (thr == 0 || r.x[e] >= thr) ? 1 : 0;
            mask[row + k] = kept;
            dst[row + k] = from_f32<T>(kept ? s * to_f32<S>(src[row + k]) : 0.0f);
        }
    }
}

// dsrc = dx * mask * s (the input gradient through the Case-I dropout)
__global__ void __launch_bounds__(256) k_case1_undrop(const float* dx, const uint8_t* mask, float* dsrc, long n,
                                                      float s) {
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256)
        dsrc[i] = mask[i] ? s * dx[i] : 0.0f;
}

// ---------------------------------------------------------------------------
// Output head of a language model (pre-FC output dropout, FC layer, softmax
// cross-entropy).  The FC products run on the input-product, dX and weight-
// gradient kernels above (K = the LSTM output width, G = the vocabulary);
// these kernels prepare their operands.

// y [T][B][F] f32 -> yb [T][B][F] and ybT [T][F][BP] in the compute type
// (rows b >= B of ybT are zero).  grid (ceil(F/32), BP/32, T), block 256.
template <typename T>
__global__ void __launch_bounds__(256) k_head_prep(const float* y, T* yb, T* ybT, int B, int F, int BP) {
    __shared__ float tile[32][33];
    const int f0 = blockIdx.x * 32, b0 = blockIdx.y * 32, t = blockIdx.z;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int r = ty; r < 32; r += 8) {
        const int b = b0 + r, f = f0 + tx;
        float v = 0.0f;
        if (b < B && f < F) {
            v = y[((size_t)t * B + b) * F + f];
            yb[((size_t)t * B + b) * F + f] = from_f32<T>(v);
        }
        tile[r][tx] = v;
    }
    __syncthreads();
    for (int r = ty; r < 32; r += 8) {
        const int f = f0 + r, b = b0 + tx;
        if (f < F) ybT[((size_t)t * F + f) * BP + b] = from_f32<T>(tile[tx][r]);
    }
}

__device__ __forceinline__ bool ce_row_valid(const int32_t* tgt, const int32_t* lengths, int t, int b, int B, int V) {
    const int g = tgt[(size_t)t * B + b];
    return g >= 0 && g < V && (!lengths || t < lengths[b]);
}

// fixed-order sum / maximum over a 256-thread block (wave shuffles, then the
// four wave results in order); every thread gets the result
__device__ __forceinline__ float block_max256(float v, float* red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return ((red[0] + red[1]) + red[2]) + red[3];
}

// Per row (t, b) of the logits: lse = log sum_v exp z_v (a pass for the
// maximum, a pass for the sum; 16-byte loads, four in flight per thread),
// the row's loss lse - z[target] and whether it counts.  grid T*B, block 256.
__global__ void __launch_bounds__(256) k_ce_rows(const float* z, const int32_t* tgt, const int32_t* lengths, int B,
                                                 int V, float* lse, float* rowloss, float* rowok) {
    __shared__ float red[4];
    const long row = blockIdx.x;
    const int t = (int)(row / B), b = (int)(row % B);
    const float4* z4 = (const float4*)(z + row * V);   // V is a multiple of 4
    const int n4 = V >> 2, tid = threadIdx.x;
    float m = -INFINITY;
    for (int i0 = tid; i0 < n4; i0 += 1024) {
        float4 q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + 256 * u;
            q[u] = i < n4 ? z4[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) m = fmaxf(m, fmaxf(fmaxf(q[u].x, q[u].y), fmaxf(q[u].z, q[u].w)));
    }
    const float M = block_max256(m, red);
    float sum = 0.0f;
    for (int i0 = tid; i0 < n4; i0 += 1024) {
        float4 q[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int i = i0 + 256 * u;
            q[u] = i < n4 ? z4[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
            sum += ((expf(q[u].x - M) + expf(q[u].y - M)) + expf(q[u].z - M)) + expf(q[u].w - M);
    }
    const float S = block_sum256(sum, red);
    if (tid == 0) {
        const float l = M + logf(S);
        const bool ok = ce_row_valid(tgt, lengths, t, b, B, V);
        lse[row] = l;
        rowloss[row] = ok ? l - z[row * V + tgt[row]] : 0.0f;
        rowok[row] = ok ? 1.0f : 0.0f;
    }
}

// loss = sum of the row losses / N, ninv = 1/N (0 when N = 0), N = rows that
// count; a fixed summation order.  One workgroup of 256.
__global__ void __launch_bounds__(256) k_ce_final(const float* rowloss, const float* rowok, long n, float* loss,
                                                  float* ninv) {
    __shared__ float sl[256], sn[256];
    float a = 0.0f, c = 0.0f;
    for (long i = threadIdx.x; i < n; i += 256) {
        a += rowloss[i];
        c += rowok[i];
    }
    sl[threadIdx.x] = a;
    sn[threadIdx.x] = c;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (threadIdx.x < h) {
            sl[threadIdx.x] += sl[threadIdx.x + h];
            sn[threadIdx.x] += sn[threadIdx.x + h];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const float N = sn[0];
        loss[0] = N > 0.0f ? sl[0] / N : 0.0f;
        ninv[0] = N > 0.0f ? 1.0f / N : 0.0f;
    }
}

// 8 consecutive values to 16-byte-aligned memory in the compute type, as
// whole 16-byte stores
__device__ __forceinline__ void st8(bf16* dst, const float* v) {
    uint32_t w[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = (uint32_t)f2bf(v[2 * q]) | ((uint32_t)f2bf(v[2 * q + 1]) << 16);
    *(uint4*)dst = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void st8(float* dst, const float* v) {
    ((float4*)dst)[0] = make_float4(v[0], v[1], v[2], v[3]);
    ((float4*)dst)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// dz = (softmax(z) - onehot(target)) / N on rows that count, 0 elsewhere,
// written in the compute type twice: fragment-major per t (the A operand of
// the dX product) and transposed [T][V][BP] (the weight-gradient operand).
// grid (ceil(V/64), T), block 256: a workgroup owns 64 columns of one t and
// walks the rows 32 at a time through an LDS tile.
template <typename T>
__global__ void __launch_bounds__(256) k_ce_grad(const float* z, const int32_t* tgt, const int32_t* lengths,
                                                 const float* lse, const float* ninv, int B, int V, int BP,
                                                 int mtiles, T* da, T* daT) {
    __shared__ float tile[32][65];
    const int v0 = blockIdx.x * 64, t = blockIdx.y;
    const int tid = threadIdx.x;
    const float sc = ninv[0];
    const int nchunk = (V + 31) / 32;
    const size_t das = (size_t)nchunk * mtiles * 512;
    T* dat = da + (size_t)t * das;
    __shared__ int rtgt[32];                   // target of each row of the block, -1 if the row does not count
    __shared__ float rlse[32];
    for (int b0 = 0; b0 < BP; b0 += 32) {
        if (tid < 32) {
            const int b = b0 + tid;
            const bool ok = b < B && ce_row_valid(tgt, lengths, t, b, B, V);
            rtgt[tid] = ok ? tgt[(size_t)t * B + b] : -1;
            rlse[tid] = ok ? lse[(size_t)t * B + b] : 0.0f;
        }
        __syncthreads();
        const int v = v0 + (tid & 63);
        float zv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {              // independent loads, all in flight
            const int r = (tid >> 6) + 4 * i;
            zv[i] = (rtgt[r] >= 0 && v < V) ? z[((size_t)t * B + b0 + r) * V + v] : 0.0f;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = (tid >> 6) + 4 * i;
            tile[r][tid & 63] = (rtgt[r] >= 0 && v < V) ? (expf(zv[i] - rlse[r]) - (v == rtgt[r] ? 1.0f : 0.0f)) * sc
                                                        : 0.0f;
        }
        __syncthreads();
        {   // transposed: thread -> column v0 + tid/4, rows 8*(tid%4) .. +7
            const int v = v0 + (tid >> 2), r0 = 8 * (tid & 3);
            if (v < V) {
                float o[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) o[e] = tile[r0 + e][tid >> 2];
                st8(daT + ((size_t)t * V + v) * BP + b0 + r0, o);
            }
        }
        {   // fragment-major: 2 chunks x 2 row tiles, one 16x32 fragment per wave
            const int f = tid >> 6, lane = tid & 63;
            const int cc = f & 1, mm = f >> 1;
            const int c = (v0 >> 5) + cc, mt = (b0 >> 4) + mm;
            if (c < nchunk && mt < mtiles) {
                const int r = 16 * mm + (lane & 15), k0 = 32 * cc + 8 * (lane >> 4);
                float o[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) o[e] = tile[r][k0 + e];
                st8(dat + frag_lane_off(c, mt, lane, mtiles), o);
            }
        }
        __syncthreads();
    }
}

// MSE loss gradient (a loss of the synthetic workloads).
__device__ __forceinline__ float nvalid_rows(const int32_t* lengths, int B, int T) {
    if (!lengths) return (float)B * T;
    float s = 0.f;
    for (int b = 0; b < B; ++b) {
        int l = lengths[b];
        l = l < 0 ? 0 : (l > T ? T : l);
        s += (float)l;
    }
    return s;
}
__global__ void __launch_bounds__(256) k_mse(const float* y, const float* tg, const int32_t* lengths,
                                             float* dy, float* partial, int T, int B, int F) {
    __shared__ float red[256];
    const float N = nvalid_rows(lengths, B, T) * (float)F;
    const float inv = N > 0.f ? 2.0f / N : 0.0f;
    // a row (t, b) per workgroup at a time, its features over the threads
    // (16 bytes each when the rows allow it): no per-element division
    const int nrows = T * B;
    const bool vec = (F & 3) == 0 && ((reinterpret_cast<uintptr_t>(y) | reinterpret_cast<uintptr_t>(tg) |
                                       reinterpret_cast<uintptr_t>(dy)) & 15) == 0;
    float acc = 0.f;
    for (int r = blockIdx.x; r < nrows; r += gridDim.x) {
        const int t = r / B, b = r - t * B;
        const bool valid = !lengths || t < lengths[b];
        const size_t o = (size_t)r * F;
        if (vec) {
            for (int f = 4 * threadIdx.x; f < F; f += 4 * blockDim.x) {
                const float4 yv = *(const float4*)(y + o + f), tv = *(const float4*)(tg + o + f);
                const float4 d = valid ? make_float4(yv.x - tv.x, yv.y - tv.y, yv.z - tv.z, yv.w - tv.w)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
                *(float4*)(dy + o + f) = make_float4(inv * d.x, inv * d.y, inv * d.z, inv * d.w);
                acc += d.x * d.x + d.y * d.y + d.z * d.z + d.w * d.w;
            }
        } else {
            for (int f = threadIdx.x; f < F; f += blockDim.x) {
                const float d = valid ? y[o + f] - tg[o + f] : 0.0f;
                dy[o + f] = inv * d;
                acc += d * d;
            }
        }
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}
__global__ void __launch_bounds__(256) k_mse_final(const float* partial, int np, const int32_t* lengths,
                                                   float* loss, int T, int B, int F) {
    __shared__ float red[256];
    float acc = 0.f;
    for (int i = threadIdx.x; i < np; i += blockDim.x) acc += partial[i];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const float N = nvalid_rows(lengths, B, T) * (float)F;
        *loss = N > 0.f ? red[0] / N : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// Kernel timer (instrumentation): HIP event pairs around the launches of one
// kernel class.
enum KernelId { KID_NONE = -1, KID_MASK, KID_TRANS, KID_FX, KID_STEP, KID_BWD, KID_DX, KID_WGRAD, KID_FWDP, KID_BWDP,
                KID_EMB, KID_CE, KID_COUNT };
static const char* const kKernelNames[KID_COUNT] = {"mask_build", "transpose", "fx", "step", "bwd", "dx", "wgrad",
                                                    "fwd_persist", "bwd_persist", "emb_grad",
                                                    "ce"};
static int g_timer_kid = KID_NONE;
static std::vector<hipEvent_t> g_ev_pool;
static size_t g_ev_used = 0;

static hipEvent_t timer_event() {
    if (g_ev_used == g_ev_pool.size()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        g_ev_pool.push_back(e);
    }
    return g_ev_pool[g_ev_used++];
}

// Event pair for a launch of kernel class kid, or false if its timer is off.
bool timer_pair(int kid, hipEvent_t* e0, hipEvent_t* e1) {
    if (g_timer_kid != kid) return false;
    *e0 = timer_event();
    *e1 = timer_event();
    return *e0 && *e1;
}

// Returns the last pair handed out (its launch did not happen).
void timer_unpair() {
    if (g_ev_used >= 2) g_ev_used -= 2;
}

int kernel_timer_start(const char* name) {
    for (int i = 0; i < KID_COUNT; ++i)
        if (name && strcmp(name, kKernelNames[i]) == 0) {
            g_timer_kid = i;
            g_ev_used = 0;
            return 0;
        }
    return -1;
}
int kernel_timer_stop(double* total_ms, int64_t* launches) {
    g_timer_kid = KID_NONE;
    double tot = 0.0;
    int64_t n = 0;
    if (g_ev_used >= 2) {
        if (hipEventSynchronize(g_ev_pool[g_ev_used - 1]) != hipSuccess) return -1;
        for (size_t i = 0; i + 1 < g_ev_used; i += 2) {
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, g_ev_pool[i], g_ev_pool[i + 1]) != hipSuccess) return -1;
            tot += ms;
            ++n;
        }
    }
    g_ev_used = 0;
    if (total_ms) *total_ms = tot;
    if (launches) *launches = n;
    return 0;
}

// Launch a kernel; while the timer is on for its class, the launch carries
// a start/stop event pair (timestamps of the dispatch itself).
template <typename... KArgs, typename... Args>
static void launch_k(int kid, void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shm, hipStream_t st,
                     Args... args) {
    if (g_timer_kid == kid) {
        hipEvent_t e0 = timer_event(), e1 = timer_event();
        if (e0 && e1) {
            hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)shm, st, e0, e1, 0, args...);
            return;
        }
    }
    kernel<<<grid, block, shm, st>>>(args...);
}
static inline int xcd_grid(int ntiles) { return NXCD * ((ntiles + NXCD - 1) / NXCD); }

// ---------------------------------------------------------------------------
// Launchers (host).
static inline int nblk(long n, int bs, int cap = 4096) {
    long g = (n + bs - 1) / bs;
    if (g < 1) g = 1;
    return (int)(g > cap ? cap : g);
}

void launch_mask_build(const MaskArgs& a, int sites, hipStream_t st) {
    launch_k(KID_MASK, k_mask_build, dim3(a.T, sites), dim3(256), 0, st, a);
}
void launch_fx_big(const FxArgs& a, hipStream_t st, hipEvent_t e0, hipEvent_t e1);
void launch_dx_big(const DxArgs& a, hipStream_t st, hipEvent_t e0, hipEvent_t e1);

// the transposes (and the pass initialisation) of FxArgs::tr on their own
template <typename T>
__global__ void __launch_bounds__(256) k_trans(FxArgs a) {
    __shared__ T tile[32][33];
    transpose_block<T>(a.tr, a.trN, blockIdx.x, blockIdx.y, blockIdx.z, a.tr_gx, a.tr_gy, tile);
}

template <typename T>
void launch_fx(const FxArgs& a, hipStream_t st) {
    if (sizeof(T) == 2 && a.XT) {              // large batch: the transposed input feeds the product
        if (a.tr_gz > 0) launch_k(KID_TRANS, k_trans<T>, dim3(a.tr_gx, a.tr_gy, a.tr_gz), dim3(256), 0, st, a);
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (g_timer_kid == KID_FX) { e0 = timer_event(); e1 = timer_event(); }
        launch_fx_big(a, st, e0, e1);
        return;
    }
    dim3 grid(xcd_grid((a.G + FX_NB - 1) / FX_NB), a.T, (a.B + FX_MB - 1) / FX_MB);
    if (a.tr_gz > 0) {                         // room for the transposes past y = T
        const long ntr = (long)a.tr_gx * a.tr_gy * a.tr_gz, per_y = (long)grid.x * grid.z;
        grid.y += (unsigned)((ntr + per_y - 1) / per_y);
    }
    if (a.dense) launch_k(KID_FX, k_fx<T, true>, grid, dim3(256), 0, st, a);
    else launch_k(KID_FX, k_fx<T, false>, grid, dim3(256), 0, st, a);
}
template <typename T>
void launch_step(const StepArgs& a, int D, hipStream_t st) {
    if (a.H > 1024)
        launch_k(KID_STEP, k_step<T, 2>, dim3(xcd_grid((a.H + 7) / 8), (a.B + 31) / 32, D), dim3(1024), 0, st, a);
    else
        launch_k(KID_STEP, k_step<T, 1>, dim3(xcd_grid((a.H + 3) / 4), (a.B + 63) / 64, D), dim3(1024), 0, st, a);
}
template <typename T>
void launch_bwd(const BwdArgs& a, int D, hipStream_t st) {
    const int nx = (a.has_next ? 2 : 1) * NXCD * a.tps;
    launch_k(KID_BWD, k_bwd<T>, dim3(nx, (a.B + 63) / 64, D), dim3(1024), 0, st, a);
}
template <typename T>
void launch_dx(const DxArgs& a, int K, hipStream_t st) {
    if (sizeof(T) == 2 && a.big) {
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (g_timer_kid == KID_DX) { e0 = timer_event(); e1 = timer_event(); }
        launch_dx_big(a, st, e0, e1);
        return;
    }
    const dim3 grid(NXCD * a.tps * 4 * ((a.T + 3) / 4), 1, (a.B + 63) / 64);
    if (a.B <= 16) launch_k(KID_DX, k_dx<T, 1>, grid, dim3(256), 0, st, a);
    else if (a.B <= 32) launch_k(KID_DX, k_dx<T, 2>, grid, dim3(256), 0, st, a);
    else launch_k(KID_DX, k_dx<T, 4>, grid, dim3(256), 0, st, a);
}
void launch_wgrad_big(const WgBatch& b, hipStream_t st, hipEvent_t e0, hipEvent_t e1);
void launch_wgrad_gemm(const WgBatch& b, hipStream_t st, hipEvent_t e0, hipEvent_t e1);
int setup_big_attributes();
// LSTM_SD_WGRAD_GEMM=0: the large-batch weight gradients on the row-sparse
// kernel (per-step gathered rows) instead of the mask-multiplied GEMM
static bool use_wgrad_gemm() {
    const char* v = getenv("LSTM_SD_WGRAD_GEMM");
    return !(v && v[0] == '0');
}

// LSTM_SD_WGRAD_STAGED=0 keeps row-sparse problems on the unstaged kernel
static bool use_wgrad_staged() {
    const char* v = getenv("LSTM_SD_WGRAD_STAGED");
    return !(v && v[0] == '0');
}
// Whether a row-sparse problem (bf16, batch <= 32) runs on the full kernel
// with its rows times the mask byte instead of the row-sparse scatter.  At a
// batch this small a step's products are nearly free, while the scatter
// pays, at every step, a chain of dependent reads (keep-list range, entries,
// rows) and an LDS read-modify-write of every kept row; measured at hidden
// 650 and 256 (batch 20 and 32) and at the AWD-LSTM shape, the full kernel
// is faster at every rate from 0.3 to 0.9, so it is the default there.
// LSTM_SD_WGRAD_ROWSPARSE=1 takes the scatter.
static bool wgrad_as_full() {
    const char* v = getenv("LSTM_SD_WGRAD_ROWSPARSE");
    return !(v && v[0] == '1');
}

template <typename T>
void launch_wgrad(const WgBatch& b, hipStream_t st) {
    if (b.np == 0) return;
    // bf16 past 32 batch rows: one GEMM per problem over every (step, batch
    // row) pair, rows times the mask byte; or (LSTM_SD_WGRAD_GEMM=0) the
    // large-batch row-sparse kernel where it applies
    if (sizeof(T) == 2 && (b.big || b.p[0].B > 32) && (use_wgrad_gemm() || b.big)) {
        hipEvent_t e0 = nullptr, e1 = nullptr;
        if (g_timer_kid == KID_WGRAD) { e0 = timer_event(); e1 = timer_event(); }
        if (use_wgrad_gemm()) launch_wgrad_gemm(b, st, e0, e1);
        else launch_wgrad_big(b, st, e0, e1);
        return;
    }
    WgBatch bs = b;
    const WgArgs& a = bs.p[0];                 // the problems share G, B and the mode
    const int ncb = (a.G + WG_NB - 1) / WG_NB;  // column blocks (wg_slot: 8 XCDs x 8 slices each)
    const dim3 grid(NXCD * NXCD * ((ncb + NXCD - 1) / NXCD), 1, bs.np);
    size_t lds = 0;
    bool multi = a.B > 32;                     // builds with the extra loops (batch chunks, tile rounds)
    for (int i = 0; i < bs.np; ++i) {
        WgArgs& p = bs.p[i];
        p.staged = p.fullmask = 0;
        if (p.full) {
            if (sizeof(T) == 2 && p.B <= 32 && use_wgrad_staged()) {
                p.staged = 1;
                lds = std::max(lds, WFS_LDS);
            } else lds = std::max(lds, wgrad_full_lds_bytes<T>());
            continue;
        }
        if (sizeof(T) == 2 && p.B <= 32 && use_wgrad_staged() && wgrad_as_full()) {
            p.full = p.staged = p.fullmask = 1;
            lds = std::max(lds, WFS_LDS);
            continue;
        }
        if (sizeof(T) == 2 && p.B <= 32 && wgs_rows(p.K) <= WGS_MAX_ROWS && wgs_lds_bytes(p.K, p.T) <= WGS_MAX_LDS &&
            use_wgrad_staged()) {
            p.staged = 1;
            lds = std::max(lds, wgs_lds_bytes(p.K, p.T));
            continue;
        }
        lds = std::max(lds, wgrad_lds_bytes<T>(p.K));
        multi = multi || (p.K + NSEG - 1) / NSEG > 16 * (WgTiles<T>::N / 2);
    }
    const dim3 blk(128 * WG_NWV);
    bool all_fs = sizeof(T) == 2;
    for (int i = 0; i < bs.np; ++i) all_fs = all_fs && bs.p[i].full && bs.p[i].staged;
    if (all_fs) {
        const dim3 bfs(WFS_FS_THREADS);
        if (a.dense) launch_k(KID_WGRAD, k_wgrad_fs<true>, grid, bfs, WFS_LDS, st, bs);
        else launch_k(KID_WGRAD, k_wgrad_fs<false>, grid, bfs, WFS_LDS, st, bs);
        return;
    }
    if (a.dense) {
        if (multi) launch_k(KID_WGRAD, k_wgrad<T, true, true>, grid, blk, lds, st, bs);
        else launch_k(KID_WGRAD, k_wgrad<T, true, false>, grid, blk, lds, st, bs);
    } else {
        if (multi) launch_k(KID_WGRAD, k_wgrad<T, false, true>, grid, blk, lds, st, bs);
        else launch_k(KID_WGRAD, k_wgrad<T, false, false>, grid, blk, lds, st, bs);
    }
}
void launch_bwd_init(const float* dhT, const float* dcT, float* dhc, float* dcs, long n, void* da, int es, int G,
                     int mtiles, long nblocks, long das, unsigned* bar, int* err, hipStream_t st) {
    const long np = da ? nblocks * 16 * mtiles * 32 : 0;      // upper bound of the DA padding entries
    launch_k(KID_NONE, k_bwd_init, dim3(nblk(n > np ? n : np, 256)), dim3(256), 0, st, dhT, dcT, dhc, dcs, n, da, es,
             G, mtiles, nblocks, das, bar, err);
}
void launch_emb_grad(const int32_t* tokens, int N, int B, int V, const float* dx, const SiteView& nr0, int I,
                     float* d_emb, hipStream_t st) {
    launch_k(KID_EMB, k_emb_grad, dim3((V + EM_VB - 1) / EM_VB, (I + EM_CW - 1) / EM_CW), dim3(256), 0, st, tokens, N,
             B, V, dx, nr0, I, d_emb);
}
template <typename T>
void launch_head_prep(const float* y, void* yb, void* ybT, int T_, int B, int F, int BP, hipStream_t st) {
    launch_k(KID_NONE, k_head_prep<T>, dim3((F + 31) / 32, BP / 32, T_), dim3(256), 0, st, y, (T*)yb, (T*)ybT, B, F,
             BP);
}
template void launch_head_prep<float>(const float*, void*, void*, int, int, int, int, hipStream_t);
template void launch_head_prep<bf16>(const float*, void*, void*, int, int, int, int, hipStream_t);
void launch_ce_loss(const float* z, const int32_t* tgt, const int32_t* lengths, int T_, int B, int V, float* lse,
                    float* rowloss, float* rowok, float* loss, float* ninv, hipStream_t st) {
    launch_k(KID_CE, k_ce_rows, dim3((unsigned)((long)T_ * B)), dim3(256), 0, st, z, tgt, lengths, B, V, lse, rowloss,
             rowok);
    launch_k(KID_CE, k_ce_final, dim3(1), dim3(256), 0, st, (const float*)rowloss, (const float*)rowok, (long)T_ * B,
             loss, ninv);
}
template <typename T>
void launch_ce_grad(const float* z, const int32_t* tgt, const int32_t* lengths, const float* lse, const float* ninv,
                    int T_, int B, int V, int BP, int mtiles, void* da, void* daT, hipStream_t st) {
    launch_k(KID_CE, k_ce_grad<T>, dim3((V + 63) / 64, T_), dim3(256), 0, st, z, tgt, lengths, lse, ninv, B, V, BP,
             mtiles, (T*)da, (T*)daT);
}
template void launch_ce_grad<float>(const float*, const int32_t*, const int32_t*, const float*, const float*, int,
                                    int, int, int, int, void*, void*, hipStream_t);
template void launch_ce_grad<bf16>(const float*, const int32_t*, const int32_t*, const float*, const float*, int,
                                   int, int, int, int, void*, void*, hipStream_t);
void launch_case1_drop(int src_f32, int dst_bf16, const void* src, void* dst, uint8_t* mask, int T_, int B, int K,
                       uint64_t seed, uint64_t step, uint64_t sid, uint64_t thr, float s, hipStream_t st) {
    const dim3 grid(((K + 3) / 4 + 63) / 64, B, T_);
    if (src_f32 && dst_bf16)
        launch_k(KID_NONE, k_case1_drop<float, bf16>, grid, dim3(64), 0, st, (const float*)src, (bf16*)dst, mask, B, K,
                 seed, step, sid, thr, s);
    else if (src_f32)
        launch_k(KID_NONE, k_case1_drop<float, float>, grid, dim3(64), 0, st, (const float*)src, (float*)dst, mask, B,
                 K, seed, step, sid, thr, s);
    else if (dst_bf16)
        launch_k(KID_NONE, k_case1_drop<bf16, bf16>, grid, dim3(64), 0, st, (const bf16*)src, (bf16*)dst, mask, B, K,
                 seed, step, sid, thr, s);
    else
        launch_k(KID_NONE, k_case1_drop<float, float>, grid, dim3(64), 0, st, (const float*)src, (float*)dst, mask, B,
                 K, seed, step, sid, thr, s);
}
void launch_case1_undrop(const float* dx, const uint8_t* mask, float* dsrc, long n, float s, hipStream_t st) {
    launch_k(KID_NONE, k_case1_undrop, dim3(nblk(n, 256)), dim3(256), 0, st, dx, mask, dsrc, n, s);
}
void launch_mse(const float* y, const float* tg, const int32_t* lengths, float* dy, float* partial, int np,
                float* loss, int T, int B, int F, hipStream_t st) {
    launch_k(KID_NONE, k_mse, dim3(np), dim3(256), 0, st, y, tg, lengths, dy, partial, T, B, F);
    launch_k(KID_NONE, k_mse_final, dim3(1), dim3(256), 0, st, (const float*)partial, np, lengths, loss, T, B, F);
}

static int g_attr_done = 0;
int setup_kernel_attributes() {
    if (g_attr_done) return 0;
    const int lds = 160 * 1024 - 1024;     // (the kernels also hold up to 1 KB of static LDS)
    const void* fns[8] = {(const void*)k_wgrad<float, false, false>, (const void*)k_wgrad<bf16, false, false>,
                          (const void*)k_wgrad<float, true, false>, (const void*)k_wgrad<bf16, true, false>,
                          (const void*)k_wgrad<float, false, true>, (const void*)k_wgrad<bf16, false, true>,
                          (const void*)k_wgrad<float, true, true>, (const void*)k_wgrad<bf16, true, true>};
    for (const void* f : fns)
        if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess) return LSTM_SD_EHIP;
    if (setup_big_attributes()) return LSTM_SD_EHIP;
    g_attr_done = 1;
    return 0;
}

#define LSD_INST(T)                                                                         \
    template void launch_fx<T>(const FxArgs&, hipStream_t);                                 \
    template void launch_step<T>(const StepArgs&, int, hipStream_t);                        \
    template void launch_bwd<T>(const BwdArgs&, int, hipStream_t);                          \
    template void launch_dx<T>(const DxArgs&, int, hipStream_t);                            \
    template void launch_wgrad<T>(const WgBatch&, hipStream_t);                             \

LSD_INST(float)
LSD_INST(bf16)

}  // namespace lsd
