// HIP kernels (gfx950, wave64) of the structured-dropout LSTM step.
//
// Every product runs on MFMA 16x16x32 tiles (bf16 inputs, fp32 accumulate;
// the fp32 path issues the fp32 MFMA).  Operands are gathered by the keep
// lists while they are loaded, so dropped rows of the contraction are never
// read or multiplied (compact mode); in dense mode the keep lists are the
// identity and the mask zeroes the dropped operands instead.
#include <hip/hip_runtime.h>

#include "device.h"
#include "kernels.h"
#include "../../include/lstm_sd.h"

namespace lsd {

// ---------------------------------------------------------------------------
// Masks (Sec. 3.1, Case-III) and compaction into keep lists.
// grid (T, sites), block 256.
__global__ void __launch_bounds__(256) k_mask_build(MaskArgs a) {
    const int t = blockIdx.x, s = blockIdx.y, tid = threadIdx.x;
    const int K = a.K[s];
    __shared__ uint8_t sm[LSTM_SD_MAX_K];
    __shared__ int wsum[4];
    uint8_t* mrow = a.mask + ((size_t)s * a.T + t) * a.kmax;
    int32_t* krow = a.keep + ((size_t)s * a.T + t) * a.kmax;
    int32_t* prow = a.pos + ((size_t)s * a.T + t) * a.kmax;
    if (a.generate) {
        const uint64_t thr = a.thr[s];
        for (int q = tid; q < (K + 3) / 4; q += blockDim.x) {
            u64x4 c;
            c.x[0] = (uint64_t)q;
            c.x[1] = (uint64_t)t;
            c.x[2] = (uint64_t)a.sid[s];
            c.x[3] = a.step;
            u64x4 r = philox4x64_10(c, a.seed, 0ull);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                int k = 4 * q + e;
                if (k < K) {
                    uint8_t kept = (thr == 0 || r.x[e] >= thr) ? 1 : 0;
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
        if (tid == 0) a.count[(size_t)s * a.T + t] = K;
        return;
    }
    const int lane = tid & 63, w = tid >> 6;
    int base = 0;
    for (int k0 = 0; k0 < K; k0 += 256) {
        const int k = k0 + tid;
        const int f = (k < K) ? sm[k] : 0;
        const unsigned long long bal = __ballot(f);
        const int pre = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) wsum[w] = __popcll(bal);
        __syncthreads();
        int off = base;
        for (int i = 0; i < w; ++i) off += wsum[i];
        const int tot = wsum[0] + wsum[1] + wsum[2] + wsum[3];
        if (k < K) {
            if (f) { krow[off + pre] = k; prow[k] = off + pre; }
            else prow[k] = -1;
        }
        base += tot;
        __syncthreads();
    }
    if (tid == 0) a.count[(size_t)s * a.T + t] = base;
}

// ---------------------------------------------------------------------------
// FP input product, all t (Eq. 1-4, first term; Sec. 3.2 FP input sparsity).
// grid (ceil(N/64), ceil(B/32), T), block 256: WG tile 32 rows x 64 cols,
// wave w owns columns 16w..16w+15 and both 16-row tiles.
template <typename T>
__global__ void __launch_bounds__(256) k_fx(FxArgs a) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int t = blockIdx.z;
    const int m0 = blockIdx.y * 32;
    const int n = blockIdx.x * 64 + w * 16 + (lane & 15);
    const int g8 = 8 * (lane >> 4);
    const T* X = (const T*)a.X + (size_t)t * a.B * a.ldx;
    const T* W = (const T*)a.W;
    const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
    const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
    const int cnt = a.site.count[t];
    f32x4_t acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
    const int r0 = m0 + (lane & 15), r1 = r0 + 16;
    for (int kc = 0; kc < cnt; kc += 32) {
        Frag<T> fa0, fa1, fb;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int j = kc + g8 + e;
            T va0 = zero_val<T>(), va1 = zero_val<T>(), vb = zero_val<T>();
            if (j < cnt) {
                const int k = krow[j];
                if (mrow[k]) {
                    if (r0 < a.B) va0 = X[(size_t)r0 * a.ldx + k];
                    if (r1 < a.B) va1 = X[(size_t)r1 * a.ldx + k];
                }
                if (n < a.N) vb = W[(size_t)k * a.N + n];
            }
            fa0.v[e] = va0; fa1.v[e] = va1; fb.v[e] = vb;
        }
        mma_16x16x32(fa0, fb, acc0);
        mma_16x16x32(fa1, fb, acc1);
    }
    if (n < a.N) {
        const float bn = a.bias[n];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int row = m0 + acc_row(lane, r);
            if (row < a.B) a.Gx[((size_t)t * a.B + row) * a.N + n] = a.s * acc0[r] + bn;
            row += 16;
            if (row < a.B) a.Gx[((size_t)t * a.B + row) * a.N + n] = a.s * acc1[r] + bn;
        }
    }
}

// ---------------------------------------------------------------------------
// One recurrent forward step (Eq. 1-6), fused with the gate pointwise.
// grid (ceil(H/4), 1, D), block 256.  A workgroup owns 4 hidden units and
// therefore the 16 gate columns {g*H + u}; the contraction over the kept
// recurrent neurons is split over the 4 waves and reduced in LDS.
template <typename T>
__global__ void __launch_bounds__(256) k_step(StepArgs a) {
    const StepDir& D = a.d[blockIdx.z];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int H = a.H, G = 4 * H, B = a.B;
    const int u0 = blockIdx.x * 4;
    const int c = lane & 15;                        // tile column
    const int ucol = u0 + (c & 3);
    const int gcol = (c >> 2) * H + ucol;           // gate column in [0, 4H)
    const bool colok = ucol < H;
    const int g8 = 8 * (lane >> 4);
    const T* hp = (const T*)D.hprev;
    const T* U = (const T*)D.U;
    const int cnt = *D.count;
    __shared__ float red[4][64][17];
    for (int mg = 0; mg < B; mg += 64) {
        f32x4_t acc[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0, 0, 0, 0};
        for (int kc = 32 * w; kc < cnt; kc += 128) {
            Frag<T> fb;
            int kk[8];
            bool kv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int j = kc + g8 + e;
                kv[e] = j < cnt;
                kk[e] = kv[e] ? D.keep[j] : 0;
                if (kv[e] && !D.mask[kk[e]]) kv[e] = false;
                fb.v[e] = (kv[e] && colok) ? U[(size_t)kk[e] * G + gcol] : zero_val<T>();
            }
#pragma unroll
            for (int mt = 0; mt < 4; ++mt) {
                const int row = mg + mt * 16 + (lane & 15);
                if (mg + mt * 16 >= B) break;
                Frag<T> fa;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    fa.v[e] = (kv[e] && row < B) ? hp[(size_t)row * H + kk[e]] : zero_val<T>();
                mma_16x16x32(fa, fb, acc[mt]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[w][mt * 16 + acc_row(lane, r)][c] = acc[mt][r];
        __syncthreads();
        // pointwise: thread -> (row, unit)
        {
            const int rr = threadIdx.x >> 2, uu = threadIdx.x & 3;
            const int b = mg + rr, u = u0 + uu;
            if (b < B && u < H) {
                float pre[4];
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int cc = g * 4 + uu;
                    float v = red[0][rr][cc] + red[1][rr][cc] + red[2][rr][cc] + red[3][rr][cc];
                    pre[g] = a.s * v + D.gx[(size_t)b * G + g * H + u];
                }
                const float ig = 1.0f / (1.0f + expf(-pre[0]));
                const float fg = 1.0f / (1.0f + expf(-pre[1]));
                const float gg = tanhf(pre[2]);
                const float og = 1.0f / (1.0f + expf(-pre[3]));
                const float cp = D.cT[(size_t)b * H + u];
                const float cn = fg * cp + ig * gg;
                const float hn = og * tanhf(cn);
                const bool valid = (a.lengths == nullptr) || (D.t < a.lengths[b]);
                float* gt = D.gates + (size_t)b * G;
                gt[u] = ig; gt[H + u] = fg; gt[2 * H + u] = gg; gt[3 * H + u] = og;
                D.cres[(size_t)b * H + u] = valid ? cn : cp;
                ((T*)D.hrec)[(size_t)b * H + u] = valid ? from_f32<T>(hn) : hp[(size_t)b * H + u];
                if (valid) {
                    D.cT[(size_t)b * H + u] = cn;
                    D.hT[(size_t)b * H + u] = hn;
                }
                if (D.y) D.y[(size_t)b * a.ldy + u] = valid ? hn : 0.0f;
                if (D.ybuf) ((T*)D.ybuf)[(size_t)b * a.ldy + u] = valid ? from_f32<T>(hn) : zero_val<T>();
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Backward pointwise of one step (Eq. 7-9 plus the activation derivatives),
// and the per-step bias-gradient partial sum over the batch.
// grid (ceil(H/16), 1, D), block 256: thread -> unit tid%16, rows tid/16 + 16i.
template <typename T>
__global__ void __launch_bounds__(256) k_bwd_pw(BwdPwArgs a) {
    const BwdPwDir& D = a.d[blockIdx.z];
    const int H = a.H, G = 4 * H, B = a.B;
    const int uu = threadIdx.x & 15, rg = threadIdx.x >> 4;
    const int u = blockIdx.x * 16 + uu;
    float dbs[4] = {0, 0, 0, 0};
    if (u < H) {
        for (int b = rg; b < B; b += 16) {
            const bool valid = (a.lengths == nullptr) || (D.t < a.lengths[b]);
            float dh = D.dhc[(size_t)b * H + u];
            if (D.dhrec) {
                const int p = D.rhpos[u];
                if (p >= 0) dh += D.dhrec[(size_t)b * H + p];
            }
            if (valid) {
                if (D.dy) dh += D.dy[(size_t)b * a.ldy + u];
                if (D.dxc) {
                    const int p = D.dxpos[u];
                    if (p >= 0) dh += D.dxc[(size_t)b * a.lddx + p];
                }
            }
            const float* gt = D.gates + (size_t)b * G;
            float da0 = 0.f, da1 = 0.f, da2 = 0.f, da3 = 0.f;
            const float dcin = D.dcs[(size_t)b * H + u];
            if (valid) {
                const float ig = gt[u], fg = gt[H + u], gg = gt[2 * H + u], og = gt[3 * H + u];
                const float ct = D.cres[(size_t)b * H + u];
                const float cp = D.cprev[(size_t)b * H + u];
                const float tc = tanhf(ct);
                const float dout = dh * tc;                           // Eq. 7
                const float dc = dh * og * (1.0f - tc * tc) + dcin;   // Eq. 7
                const float df = dc * cp, di = dc * gg, dg = dc * ig; // Eq. 8-9
                da0 = di * ig * (1.0f - ig);
                da1 = df * fg * (1.0f - fg);
                da2 = dg * (1.0f - gg * gg);
                da3 = dout * og * (1.0f - og);
                D.dcs[(size_t)b * H + u] = dc * fg;                   // Eq. 8
                D.dhc[(size_t)b * H + u] = 0.0f;
            } else {
                D.dhc[(size_t)b * H + u] = dh;                        // frozen row
            }
            T* dar = (T*)D.da + (size_t)b * G;
            dar[u] = from_f32<T>(da0);
            dar[H + u] = from_f32<T>(da1);
            dar[2 * H + u] = from_f32<T>(da2);
            dar[3 * H + u] = from_f32<T>(da3);
            dbs[0] += da0; dbs[1] += da1; dbs[2] += da2; dbs[3] += da3;
        }
    }
    __shared__ float red[16][4][16];
#pragma unroll
    for (int g = 0; g < 4; ++g) red[rg][g][uu] = dbs[g];
    __syncthreads();
    if (threadIdx.x < 64) {
        const int g = threadIdx.x >> 4, q = threadIdx.x & 15;
        const int uq = blockIdx.x * 16 + q;
        if (uq < H) {
            float s = 0.f;
            for (int i = 0; i < 16; ++i) s += red[i][g][q];
            D.dbpart[g * H + uq] = s;
        }
    }
}

// ---------------------------------------------------------------------------
// Output-sparse recurrent gradient of one step (Eq. 10, Sec. 3.2 BP):
//   dhrec[b][j] = s * m * sum_n DA[b][n] U[keep[j]][n], j < count.
// grid (ceil(H/64), ceil(B/32), D), block 256; tile 32 rows x 64 kept columns.
template <typename T>
__global__ void __launch_bounds__(256) k_bwd_dh(DhArgs a) {
    const DhDir& D = a.d[blockIdx.z];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int cnt = *D.count;
    const int j0 = blockIdx.x * 64;
    if (j0 >= cnt) return;
    const int m0 = blockIdx.y * 32;
    const int j = j0 + w * 16 + (lane & 15);
    const int g8 = 8 * (lane >> 4);
    const T* DA = (const T*)D.da;
    const T* Wk = (const T*)D.Wk;
    const int k = (j < cnt) ? D.keep[j] : -1;
    const int r0 = m0 + (lane & 15), r1 = r0 + 16;
    f32x4_t acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
    for (int nc = 0; nc < a.G; nc += 32) {
        Frag<T> fa0, fa1, fb;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int n = nc + g8 + e;
            const bool nv = n < a.G;
            fa0.v[e] = (nv && r0 < a.B) ? DA[(size_t)r0 * a.G + n] : zero_val<T>();
            fa1.v[e] = (nv && r1 < a.B) ? DA[(size_t)r1 * a.G + n] : zero_val<T>();
            fb.v[e] = (nv && k >= 0) ? Wk[(size_t)k * a.G + n] : zero_val<T>();
        }
        mma_16x16x32(fa0, fb, acc0);
        mma_16x16x32(fa1, fb, acc1);
    }
    // columns of this lane's outputs: j (acc_col = lane & 15)
    if (j < cnt) {
        const float sc = D.mask[k] ? a.s : 0.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int row = m0 + acc_row(lane, r);
            if (row < a.B) D.out[(size_t)row * a.ldo + j] = sc * acc0[r];
            row += 16;
            if (row < a.B) D.out[(size_t)row * a.ldo + j] = sc * acc1[r];
        }
    }
}

// ---------------------------------------------------------------------------
// Output-sparse input gradient, all t (Eq. 10), summed over directions:
//   dxc[t][b][j] = s * m * sum_d sum_n DA_d[t][b][n] W_d[keep_t[j]][n].
// grid (ceil(Kmax/64), ceil(B/32), T), block 256.
template <typename T>
__global__ void __launch_bounds__(256) k_dx(DxArgs a) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int t = blockIdx.z;
    const int cnt = a.site.count[t];
    const int j0 = blockIdx.x * 64;
    if (j0 >= cnt) return;
    const int m0 = blockIdx.y * 32;
    const int j = j0 + w * 16 + (lane & 15);
    const int g8 = 8 * (lane >> 4);
    const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
    const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
    const int k = (j < cnt) ? krow[j] : -1;
    const int r0 = m0 + (lane & 15), r1 = r0 + 16;
    f32x4_t acc0 = {0, 0, 0, 0}, acc1 = {0, 0, 0, 0};
    for (int d = 0; d < a.D; ++d) {
        const T* DA = (const T*)a.da[d] + (size_t)t * a.B * a.G;
        const T* Wk = (const T*)a.W[d];
        for (int nc = 0; nc < a.G; nc += 32) {
            Frag<T> fa0, fa1, fb;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int n = nc + g8 + e;
                const bool nv = n < a.G;
                fa0.v[e] = (nv && r0 < a.B) ? DA[(size_t)r0 * a.G + n] : zero_val<T>();
                fa1.v[e] = (nv && r1 < a.B) ? DA[(size_t)r1 * a.G + n] : zero_val<T>();
                fb.v[e] = (nv && k >= 0) ? Wk[(size_t)k * a.G + n] : zero_val<T>();
            }
            mma_16x16x32(fa0, fb, acc0);
            mma_16x16x32(fa1, fb, acc1);
        }
    }
    if (j < cnt) {
        const float sc = mrow[k] ? a.s : 0.0f;
        float* out = a.out + (size_t)t * a.B * a.ldo;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int row = m0 + acc_row(lane, r);
            if (row < a.B) out[(size_t)row * a.ldo + j] = sc * acc0[r];
            row += 16;
            if (row < a.B) out[(size_t)row * a.ldo + j] = sc * acc1[r];
        }
    }
}

// ---------------------------------------------------------------------------
// Row-sparse weight gradient (Eq. 11, Sec. 3.2 WG), summed over t.
// grid (ceil(G/16)), block 256, dynamic LDS K*16 floats: a workgroup owns 16
// columns of dW for every row and accumulates in LDS; at each t the kept
// rows are processed in 16-row tiles (distinct rows per tile, so waves never
// collide), and rows never kept stay exactly zero.
template <typename T>
__global__ void __launch_bounds__(256) k_wgrad(WgArgs a) {
    extern __shared__ float acc_lds[];   // [K][16]
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int n0 = blockIdx.x * 16;
    const int col = lane & 15;
    const int n = n0 + col;
    const int g8 = 8 * (lane >> 4);
    for (int i = threadIdx.x; i < a.K * 16; i += blockDim.x) acc_lds[i] = 0.0f;
    __syncthreads();
    const T* DAall = (const T*)a.da;
    for (int t = 0; t < a.T; ++t) {
        const int cnt = a.site.count[t];
        const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
        const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
        const T* act;
        if (a.act_first && t == a.t_first) act = (const T*)a.act_first;
        else act = (const T*)a.act + (long)(t + a.act_shift) * a.act_tstride;
        const T* DA = DAall + (size_t)t * a.B * a.G;
        for (int jt = w; jt * 16 < cnt; jt += 4) {
            const int j = jt * 16 + (lane & 15);        // A row of this lane
            int k = -1;
            if (j < cnt) { k = krow[j]; if (!mrow[k]) k = -1; }
            f32x4_t acc = {0, 0, 0, 0};
            for (int bc = 0; bc < a.B; bc += 32) {
                Frag<T> fa, fb;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int b = bc + g8 + e;
                    const bool bv = b < a.B;
                    fa.v[e] = (bv && k >= 0) ? act[(size_t)b * a.act_ld + k] : zero_val<T>();
                    fb.v[e] = (bv && n < a.G) ? DA[(size_t)b * a.G + n] : zero_val<T>();
                }
                mma_16x16x32(fa, fb, acc);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int jr = jt * 16 + acc_row(lane, r);
                if (jr < cnt) {
                    const int kr = krow[jr];
                    acc_lds[kr * 16 + col] += a.s * acc[r];
                }
            }
        }
        __syncthreads();
    }
    for (int i = threadIdx.x; i < a.K * 16; i += blockDim.x) {
        const int kr = i >> 4, cc = i & 15;
        if (n0 + cc < a.G) a.dW[(size_t)kr * a.G + n0 + cc] = acc_lds[i];
    }
}

// ---------------------------------------------------------------------------
// Small elementwise kernels.

// hT <- h0 (as float), cT <- c0
template <typename T>
__global__ void k_fwd_init(const T* h0, const float* c0, float* hT, float* cT, long n) {
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        hT[i] = to_f32<T>(h0[i]);
        cT[i] = c0[i];
    }
}

// carries <- dhT/dcT slices (or zero) for D directions of one layer
__global__ void k_bwd_init(const float* dhT, const float* dcT, float* dhc, float* dcs, long n) {
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        dhc[i] = dhT ? dhT[i] : 0.0f;
        dcs[i] = dcT ? dcT[i] : 0.0f;
    }
}

// dh0 = (expanded last recurrent gradient) + carry, dc0 = cell carry
__global__ void k_bwd_final(FinalArgs a) {
    const FinalDir& D = a.d[blockIdx.y];
    const long n = (long)a.B * a.H;
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        const int b = (int)(i / a.H), u = (int)(i % a.H);
        float v = D.dhc[i];
        if (D.dhrec) {
            const int p = D.rhpos[u];
            if (p >= 0) v += D.dhrec[(size_t)b * a.H + p];
        }
        D.dh0[i] = v;
        D.dc0[i] = D.dcs[i];
    }
}

// dx[t][b][k] = dxc[t][b][pos_t[k]] (0 where the neuron is not listed)
__global__ void k_expand(const float* dxc, int ldc, SiteView site, float* dx, int B, int K, int T) {
    const long n = (long)T * B * K;
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        const int k = (int)(i % K);
        const long tb = i / K;
        const int t = (int)(tb / B);
        const int p = site.pos[(size_t)t * site.kmax + k];
        dx[i] = p >= 0 ? dxc[tb * ldc + p] : 0.0f;
    }
}

// db[n] = sum_t dbpart[t][n]
__global__ void k_db(const float* dbpart, float* db, int G, int T) {
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= G) return;
    float s = 0.f;
    for (int t = 0; t < T; ++t) s += dbpart[(size_t)t * G + n];
    db[n] = s;
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
    const long n = (long)T * B * F;
    float acc = 0.f;
    for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
        const long tb = i / F;
        const int t = (int)(tb / B), b = (int)(tb % B);
        const bool valid = !lengths || t < lengths[b];
        const float d = valid ? y[i] - tg[i] : 0.0f;
        dy[i] = inv * d;
        acc += d * d;
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
// Launchers (host).
static inline int nblk(long n, int bs, int cap = 4096) {
    long g = (n + bs - 1) / bs;
    if (g < 1) g = 1;
    return (int)(g > cap ? cap : g);
}

void launch_mask_build(const MaskArgs& a, int sites, hipStream_t st) {
    hipLaunchKernelGGL(k_mask_build, dim3(a.T, sites), dim3(256), 0, st, a);
}

template <typename T>
void launch_fx(const FxArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(k_fx<T>, dim3((a.N + 63) / 64, (a.B + 31) / 32, a.T), dim3(256), 0, st, a);
}
template <typename T>
void launch_step(const StepArgs& a, int D, hipStream_t st) {
    hipLaunchKernelGGL(k_step<T>, dim3((a.H + 3) / 4, 1, D), dim3(256), 0, st, a);
}
template <typename T>
void launch_bwd_pw(const BwdPwArgs& a, int D, hipStream_t st) {
    hipLaunchKernelGGL(k_bwd_pw<T>, dim3((a.H + 15) / 16, 1, D), dim3(256), 0, st, a);
}
template <typename T>
void launch_bwd_dh(const DhArgs& a, int D, int H, hipStream_t st) {
    hipLaunchKernelGGL(k_bwd_dh<T>, dim3((H + 63) / 64, (a.B + 31) / 32, D), dim3(256), 0, st, a);
}
template <typename T>
void launch_dx(const DxArgs& a, int K, hipStream_t st) {
    hipLaunchKernelGGL(k_dx<T>, dim3((K + 63) / 64, (a.B + 31) / 32, a.T), dim3(256), 0, st, a);
}
template <typename T>
void launch_wgrad(const WgArgs& a, hipStream_t st) {
    size_t lds = (size_t)a.K * 16 * sizeof(float);
    hipLaunchKernelGGL(k_wgrad<T>, dim3((a.G + 15) / 16), dim3(256), lds, st, a);
}
template <typename T>
void launch_fwd_init(const void* h0, const float* c0, float* hT, float* cT, long n, hipStream_t st) {
    hipLaunchKernelGGL(k_fwd_init<T>, dim3(nblk(n, 256)), dim3(256), 0, st, (const T*)h0, c0, hT, cT, n);
}
void launch_bwd_init(const float* dhT, const float* dcT, float* dhc, float* dcs, long n, hipStream_t st) {
    hipLaunchKernelGGL(k_bwd_init, dim3(nblk(n, 256)), dim3(256), 0, st, dhT, dcT, dhc, dcs, n);
}
void launch_bwd_final(const FinalArgs& a, int D, hipStream_t st) {
    hipLaunchKernelGGL(k_bwd_final, dim3(nblk((long)a.B * a.H, 256), D), dim3(256), 0, st, a);
}
void launch_expand(const float* dxc, int ldc, const SiteView& s, float* dx, int B, int K, int T, hipStream_t st) {
    hipLaunchKernelGGL(k_expand, dim3(nblk((long)T * B * K, 256)), dim3(256), 0, st, dxc, ldc, s, dx, B, K, T);
}
void launch_db(const float* dbpart, float* db, int G, int T, hipStream_t st) {
    hipLaunchKernelGGL(k_db, dim3((G + 255) / 256), dim3(256), 0, st, dbpart, db, G, T);
}
void launch_mse(const float* y, const float* tg, const int32_t* lengths, float* dy, float* partial, int np,
                float* loss, int T, int B, int F, hipStream_t st) {
    hipLaunchKernelGGL(k_mse, dim3(np), dim3(256), 0, st, y, tg, lengths, dy, partial, T, B, F);
    hipLaunchKernelGGL(k_mse_final, dim3(1), dim3(256), 0, st, partial, np, lengths, loss, T, B, F);
}

static int g_attr_done = 0;
int setup_kernel_attributes() {
    if (g_attr_done) return 0;
    const int lds = 160 * 1024;
    hipError_t e1 = hipFuncSetAttribute((const void*)k_wgrad<float>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    hipError_t e2 = hipFuncSetAttribute((const void*)k_wgrad<bf16>, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e1 != hipSuccess || e2 != hipSuccess) return LSTM_SD_EHIP;
    g_attr_done = 1;
    return 0;
}

template void launch_fx<float>(const FxArgs&, hipStream_t);
template void launch_fx<bf16>(const FxArgs&, hipStream_t);
template void launch_step<float>(const StepArgs&, int, hipStream_t);
template void launch_step<bf16>(const StepArgs&, int, hipStream_t);
template void launch_bwd_pw<float>(const BwdPwArgs&, int, hipStream_t);
template void launch_bwd_pw<bf16>(const BwdPwArgs&, int, hipStream_t);
template void launch_bwd_dh<float>(const DhArgs&, int, int, hipStream_t);
template void launch_bwd_dh<bf16>(const DhArgs&, int, int, hipStream_t);
template void launch_dx<float>(const DxArgs&, int, hipStream_t);
template void launch_dx<bf16>(const DxArgs&, int, hipStream_t);
template void launch_wgrad<float>(const WgArgs&, hipStream_t);
template void launch_wgrad<bf16>(const WgArgs&, hipStream_t);
template void launch_fwd_init<float>(const void*, const float*, float*, float*, long, hipStream_t);
template void launch_fwd_init<bf16>(const void*, const float*, float*, float*, long, hipStream_t);

}  // namespace lsd
