// Products of the step at large batches (gfx950, bf16, 64 rows or more): the
// weight gradients (Eq. 11), the input products (Eq. 1-4) and the input
// gradients (Eq. 10).  At a batch of a few hundred rows every product is a
// large GEMM over gathered rows, so these kernels stage operand chunks in LDS
// for a whole workgroup (8 waves on a 128- or 256-row tile), with the loads
// issued two chunks ahead, where the small-batch kernels (one contraction
// chunk per step, operands straight from the cache) are bound by latency.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>

#include "device.h"
#include "kernels.h"
#include "../../include/lstm_sd.h"

namespace lsd {


// ---------------------------------------------------------------------------
// Weight gradient for large batches, Eq. 11:
//   dW[k][n] = s * sum_t sum_{b} act_t[b][k] da_t[b][n]
// over the steps t at which row k is kept (row-sparse), or every step with
// the mask as a multiplier (the dense comparison mode); rows never kept are
// 0.  grid (row slices of 128 x column blocks of 128, 1, problems), 512
// threads (8 waves); workgroup i runs on XCD i % 8, which takes the column
// blocks x, x+8, ... with every row slice, so one XCD's L2 holds its
// columns' DA^T of a step once for all of its slices.
// At each step the kept rows of the slice are listed in ascending order (a
// ballot over the mask bytes), and the contraction over the batch runs in
// chunks of 64 batch rows: the chunk of the listed rows of act_t^T ([K][BP])
// and of the block's 128 columns of DA_t^T ([G][BP]) are staged in LDS as
// [row][64+8] tiles (whole 16-byte pieces of each row), double buffered,
// with the loads issued two chunks ahead across step boundaries.  The
// step's product (listed rows x 128 columns) is tiled in 16x16 MFMA tiles:
// wave w takes the columns 32*(w%4) .. +31 and the row tiles w/4, w/4+2,
// .. (those past the listed count are skipped), and at the end of the step
// adds its tiles into the slice's rows of an LDS accumulator (the rows of
// one step are distinct; the positions past the count go to a spare row).
// Slice 0 also sums the bias gradient.  One launch covers every problem of
// a pass.
constexpr int WL_R = 128, WL_C = 128, WL_KC = 64, WL_P = WL_KC + 8, WL_LDC = WL_C + 4;
constexpr size_t WL_LDS = (size_t)(WL_R + 1) * WL_LDC * 4 + (size_t)2 * (WL_R + WL_C) * WL_P * 2 +
                          (size_t)4 * 2 * WL_R * 4 + 64;

__global__ void __launch_bounds__(512) k_wgrad_big(WgBatch bt) {
    extern __shared__ __align__(16) char smem[];
    const WgArgs& a = bt.p[blockIdx.z];
    const int nrs = (a.K + WL_R - 1) / WL_R, ncb = (a.G + WL_C - 1) / WL_C;
    const int xcd = blockIdx.x % 8, k8 = blockIdx.x / 8;
    const int rs = k8 % nrs, cb = xcd + 8 * (k8 / nrs);
    if (cb >= ncb) return;
    const int r0 = rs * WL_R, nrow = min(WL_R, a.K - r0), n0 = cb * WL_C;
    float* acc_lds = (float*)smem;                                        // [WL_R + 1][WL_LDC]
    bf16* As = (bf16*)(smem + (size_t)(WL_R + 1) * WL_LDC * 4);           // [2][WL_R][WL_P]
    bf16* Bs = As + 2 * WL_R * WL_P;                                      // [2][WL_C][WL_P]
    int* lrow = (int*)(Bs + 2 * WL_C * WL_P);                             // [4][WL_R] rows to load (-1: zero)
    int* trow = lrow + 4 * WL_R;                                          // [4][WL_R] accumulator rows
    int* lcount = trow + 4 * WL_R;                                        // [4]
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int B = a.B, G = a.G, T_ = a.T;
    const int nb = (B + WL_KC - 1) / WL_KC, nq = T_ * nb;               // chunks per step, in all
    const bool failed = bt.status && *bt.status != 0;
    for (int i = tid; i < (WL_R + 1) * WL_LDC; i += 512) acc_lds[i] = 0.0f;

    // the row list of step t into ring slot t % 4 (wave 0; mask bytes of
    // the step in mk0 / mk1): compact mode lists the kept rows of the slice
    // in ascending order, then -1 (loaded as zero, added into the spare
    // row); dense mode lists every row, a dropped one loaded as zero
    auto mask_load = [&](int t, uint32_t& mk0, uint32_t& mk1) {
        const uint8_t* mrow = a.site.mask + (size_t)min(t, T_ - 1) * a.site.kmax + r0;
        mk0 = mrow[min(lane, nrow - 1)];
        mk1 = mrow[min(lane + 64, nrow - 1)];
    };
    auto build = [&](int t, uint32_t mk0, uint32_t mk1) {
        int* lr = lrow + (t & 3) * WL_R;
        int* tr = trow + (t & 3) * WL_R;
        const bool k0 = t < T_ && lane < nrow && mk0 != 0;
        const bool k1 = t < T_ && lane + 64 < nrow && mk1 != 0;
        if (a.dense) {
            lr[lane] = k0 ? r0 + lane : -1;
            lr[lane + 64] = k1 ? r0 + 64 + lane : -1;
            tr[lane] = lane < nrow ? lane : WL_R;
            tr[lane + 64] = lane + 64 < nrow ? lane + 64 : WL_R;
            if (lane == 0) lcount[t & 3] = t < T_ ? nrow : 0;
            return;
        }
        const uint64_t b0 = __builtin_amdgcn_ballot_w64(k0), b1 = __builtin_amdgcn_ballot_w64(k1);
        const int c0 = __popcll(b0), n = c0 + __popcll(b1);
        const int i0 = __builtin_amdgcn_mbcnt_hi((uint32_t)(b0 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b0, 0));
        const int i1 = c0 + __builtin_amdgcn_mbcnt_hi((uint32_t)(b1 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b1, 0));
        if (k0) { lr[i0] = r0 + lane; tr[i0] = lane; }
        if (k1) { lr[i1] = r0 + 64 + lane; tr[i1] = 64 + lane; }
        if (n + lane < WL_R) { lr[n + lane] = -1; tr[n + lane] = WL_R; }
        if (n + 64 + lane < WL_R) { lr[n + 64 + lane] = -1; tr[n + 64 + lane] = WL_R; }
        if (lane == 0) lcount[t & 3] = n;
    };
    auto act_ptr = [&](int t) {
        return (a.actT_first && t == a.t_first) ? (const bf16*)a.actT_first
                                                : (const bf16*)a.actT + (long)(t + a.shift) * a.tstride;
    };
    // lists are built three steps ahead: with one chunk per step the loads
    // of step t+2 go out during step t, before its list would otherwise be
    // built
    uint32_t mk0 = 0, mk1 = 0;
    if (w == 0) {
        for (int t = 0; t < 3; ++t) {
            mask_load(t, mk0, mk1);
            build(t, mk0, mk1);
        }
        mask_load(3, mk0, mk1);                                           // (step 3's, built at step 0)
    }
    __syncthreads();

    // staging of chunk q = t * nb + c: thread -> (row slot tid/8 + 64i,
    // 16-byte piece tid%8) of A and of B; batch entries past B are zeroed
    const int sr = tid >> 3, sp = tid & 7;
    u32x4_t ra[2][2], rb[2][2];
    float dbacc[2] = {0.0f, 0.0f};
    const bool dbw = a.db && rs == 0;
    auto fetch = [&](int set, int q) {
        const bool live = q < nq;
        const int t = live ? q / nb : T_ - 1, c = live ? q % nb : 0;
        const int bq = WL_KC * c + 8 * sp;                                // first batch entry of the piece
        const __amdgpu_buffer_rsrc_t ar = buf_rsrc(act_ptr(t), (uint32_t)((size_t)a.K * a.BP * 2));
        const __amdgpu_buffer_rsrc_t br = buf_rsrc((const bf16*)a.daT + (size_t)t * G * a.BP,
                                                   (uint32_t)((size_t)G * a.BP * 2));
        const int* lr = lrow + (t & 3) * WL_R;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int r = lr[sr + 64 * i];
            const uint32_t oa = (live && r >= 0 && bq < B) ? (uint32_t)((size_t)r * a.BP + bq) * 2 : OOB_OFF;
            ra[set][i] = __builtin_amdgcn_raw_buffer_load_b128(ar, oa, 0, 0);
            const int n = n0 + sr + 64 * i;
            const uint32_t ob = (live && n < G && bq < B) ? (uint32_t)((size_t)n * a.BP + bq) * 2 : OOB_OFF;
            rb[set][i] = __builtin_amdgcn_raw_buffer_load_b128(br, ob, 0, 0);
        }
    };
    auto commit = [&](int set, int buf, int q) {
        const int c = q % nb;
        const int bq = WL_KC * c + 8 * sp;
        uint32_t m[4];
        pad_mask<bf16>(bq, B, m);                                         // (batch entries past B)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            u32x4_t x = ra[set][i], y = rb[set][i];
#pragma unroll
            for (int e = 0; e < 4; ++e) { x[e] &= m[e]; y[e] &= m[e]; }
            *(u32x4_t*)(As + ((size_t)buf * WL_R + sr + 64 * i) * WL_P + 8 * sp) = x;
            *(u32x4_t*)(Bs + ((size_t)buf * WL_C + sr + 64 * i) * WL_P + 8 * sp) = y;
            if (dbw && q < nq) {
#pragma unroll
                for (int e = 0; e < 4; ++e) dbacc[i] += __uint_as_float(y[e] << 16) + __uint_as_float(y[e] & 0xffff0000u);
            }
        }
    };

    f32x4_t acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
    const int mw = w >> 2, cw = 32 * (w & 3);
    const int cl = lane & 15, g8 = 8 * (lane >> 4);
    int cnt = lcount[0];                                                  // rows of the current step
    fetch(0, 0);
    fetch(1, 1);
    commit(0, 0, 0);
    __syncthreads();
    // chunk q (LDS buffer cur = q % 2): the loads of q+2 go out, then the
    // products; at the first chunk of a step wave 0 lists the rows of step
    // t+3 (ring slot (t+3) % 4, whose step t-1 is done), at the last the
    // step's tiles go into the accumulator
    auto chunk = [&](int q, int cur) {
        fetch(cur, q + 2);
        __builtin_amdgcn_sched_barrier(0);     // (the loads go out before anything waits)
        const int t = q / nb, c = q % nb;
        if (c == 0 && w == 0) {
            build(t + 3, mk0, mk1);
            mask_load(t + 4, mk0, mk1);
        }
        const bf16* Ab = As + (size_t)cur * WL_R * WL_P;
        const bf16* Bb = Bs + (size_t)cur * WL_C * WL_P;
#pragma unroll
        for (int ks = 0; ks < WL_KC / 32; ++ks) {
            Raw8<bf16> fb[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) raw_lds(fb[j], Bb + (size_t)(cw + 16 * j + cl) * WL_P + 32 * ks + g8);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int mt = mw + 2 * i;
                if (16 * mt >= cnt) break;                                // (uniform) row tiles past the list
                Raw8<bf16> fa;
                raw_lds(fa, Ab + (size_t)(16 * mt + cl) * WL_P + 32 * ks + g8);
#pragma unroll
                for (int j = 0; j < 2; ++j) raw_mma(fa, fb[j], acc[i][j]);
            }
        }
        if (c == nb - 1) {
            // the step's tiles into their rows: every wave's additions of
            // the step before are complete (a barrier ends every chunk)
            const int* tr = trow + (t & 3) * WL_R;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int mt = mw + 2 * i;
                if (16 * mt >= cnt) break;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float* d = acc_lds + (size_t)tr[16 * mt + acc_row(lane, r)] * WL_LDC + cw + 16 * j + cl;
                        *d += a.s * acc[i][j][r];
                    }
                    acc[i][j] = f32x4_t{0, 0, 0, 0};
                }
            }
        }
        commit(cur ^ 1, cur ^ 1, q + 1);
        __syncthreads();
        if (c == nb - 1) cnt = lcount[(t + 1) & 3];
    };
    int q = 0;
    for (; q + 1 < nq; q += 2) {
        chunk(q, 0);
        chunk(q + 1, 1);
    }
    if (q < nq) chunk(q, 0);
    __syncthreads();
    const float nan = __builtin_nanf("");
    for (int i = tid; i < nrow * WL_C; i += 512) {
        const int r = i / WL_C, c = i % WL_C;
        if (n0 + c < G) a.out[(size_t)(r0 + r) * G + n0 + c] = failed ? nan : acc_lds[r * WL_LDC + c];
    }
    if (dbw) {
        // the 8 threads of a column slot hold its partial sums over their pieces
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            float v = dbacc[i];
            v += __shfl_xor(v, 1);
            v += __shfl_xor(v, 2);
            v += __shfl_xor(v, 4);
            const int n = n0 + sr + 64 * i;
            if (sp == 0 && n < G) a.db[n] = failed ? nan : v;
        }
    }
}

// ---------------------------------------------------------------------------
// Forward input product for large batches (Eq. 1-4 input term; Sec. 3.2 FP
// input sparsity):
//   Gx_t = s * X_t[:, keep_t] W[keep_t, :] + bias
// grid (ceil(G/128), T, ceil(B/256)), 512 threads (8 waves).  A workgroup
// computes a 256-row x 128-column tile of Gx_t; wave w owns rows
// 64*(w/2) .. +63 and columns 64*(w%2) .. +63 (4 x 4 tiles of
// 16x16x32 MFMA).  The contraction runs over the keep list of t in chunks
// of 64 kept neurons: the gathered rows of the transposed input X_t^T
// ([K][ld], 256 batch columns) and of W (128 columns) are staged in LDS as
// K-major tiles (whole 16-byte pieces of each row, coalesced), double
// buffered so that chunk i+1 is in flight while chunk i is multiplied, and
// both operands' fragments are read with ds_read_b64_tr_b16 (lanes 4e..4e+3
// of a 16-lane group address row e of the group's four at columns 0, 4, 8,
// 12: lane i receives column i of the four rows).  Dropped rows of the
// dense mode and rows past the count read as zero (an offset past the
// buffer).  Rows past B and columns past G are computed and not stored.
constexpr int FB_M = 256, FB_N = 128, FB_KC = 64, FB_AP = FB_M + 16, FB_BP = FB_N + 16;
constexpr size_t FB_LDS = (size_t)2 * FB_KC * (FB_AP + FB_BP) * 2 + (size_t)(LSTM_SD_MAX_K + 2 * FB_KC) * 4;

__global__ void __launch_bounds__(512) k_fx_big(FxArgs a) {
    extern __shared__ __align__(16) char smem[];
    bf16* As = (bf16*)smem;                                  // [2][FB_KC][FB_AP]
    bf16* Bs = As + 2 * FB_KC * FB_AP;                       // [2][FB_KC][FB_BP]
    int* kidx = (int*)(Bs + 2 * FB_KC * FB_BP);              // [count]
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int t = blockIdx.y, n0 = blockIdx.x * FB_N, m0 = blockIdx.z * FB_M;
    const int K = a.K, G = a.G, B = a.B;
    const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
    const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
    const int cnt = a.site.count[t];
    // the keep list, then -1 through two chunks past the last (rows read as
    // zero: the loop fetches two chunks ahead without a condition)
    const int cpad = ((cnt + FB_KC - 1) / FB_KC + 2) * FB_KC;
    for (int j = tid; j < cpad; j += 512) kidx[j] = j >= cnt || (a.dense && !mrow[j]) ? -1 : krow[j];
    __syncthreads();
    const __amdgpu_buffer_rsrc_t xr = buf_rsrc((const bf16*)a.XT + (size_t)t * a.xt_tstride,
                                               (uint32_t)((size_t)K * a.xt_ld * 2));
    const __amdgpu_buffer_rsrc_t wr = buf_rsrc(a.W, (uint32_t)((size_t)K * G * 2));
    // staging: A rows (512 bytes of X^T) as 32 pieces, 4 per thread; B rows
    // (256 bytes of W) as 16 pieces, 2 per thread.  Chunk j goes through
    // register set j % 2: its loads are issued two chunks ahead, so each
    // has two chunks' products to arrive in
    u32x4_t ra[2][4], rb[2][2];
    // (every row index of a chunk is read first, then its six loads go out
    // back to back; absent rows take an offset past the buffer: no branch)
    const uint32_t aoff = (uint32_t)(m0 + 8 * (tid & 31)) * 2, boff = (uint32_t)(n0 + 8 * (tid & 15)) * 2;
    auto fetch = [&](int set, int kc) {
        int ka[4], kb[2];
#pragma unroll
        for (int i = 0; i < 4; ++i) ka[i] = kidx[kc + (tid >> 5) + 16 * i];
#pragma unroll
        for (int i = 0; i < 2; ++i) kb[i] = kidx[kc + (tid >> 4) + 32 * i];
        uint32_t oa[4], ob[2];
#pragma unroll
        for (int i = 0; i < 4; ++i) oa[i] = ka[i] < 0 ? OOB_OFF : (uint32_t)ka[i] * (uint32_t)(a.xt_ld * 2) + aoff;
#pragma unroll
        for (int i = 0; i < 2; ++i) ob[i] = kb[i] < 0 ? OOB_OFF : (uint32_t)kb[i] * (uint32_t)(G * 2) + boff;
#pragma unroll
        for (int i = 0; i < 4; ++i) ra[set][i] = __builtin_amdgcn_raw_buffer_load_b128(xr, oa[i], 0, 0);
#pragma unroll
        for (int i = 0; i < 2; ++i) rb[set][i] = __builtin_amdgcn_raw_buffer_load_b128(wr, ob[i], 0, 0);
    };
    auto commit = [&](int set, int buf) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = tid + 512 * i, r = q >> 5, c = q & 31;
            *(u32x4_t*)(As + ((size_t)buf * FB_KC + r) * FB_AP + 8 * c) = ra[set][i];
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int q = tid + 512 * i, r = q >> 4, c = q & 15;
            *(u32x4_t*)(Bs + ((size_t)buf * FB_KC + r) * FB_BP + 8 * c) = rb[set][i];
        }
    };
    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
    const int wr0 = 64 * (w >> 1), wc0 = 64 * (w & 1);
    const int trow = 8 * (lane >> 4) + ((lane & 15) >> 2), tcol = 4 * (lane & 3);
    const int nch = (cnt + FB_KC - 1) / FB_KC;
    fetch(0, 0);
    fetch(1, FB_KC);
    commit(0, 0);
    __syncthreads();
    // chunk ch (in LDS buffer ch % 2): the loads of ch+2 go out, the
    // products of ch, then ch+1 (loaded during ch-1) into the other buffer
    // (fetch and commit run unconditionally, past the end on zero rows: a
    // conditional load leaves the compiler unsure which loads are still in
    // flight, and it then waits for all of them before the next fetch)
    auto chunk = [&](int ch, int cur) {
        fetch(cur, (ch + 2) * FB_KC);
        __builtin_amdgcn_sched_barrier(0);     // (the loads go out before anything waits)
        const int buf = cur;
        const bf16* Ab = As + (size_t)buf * FB_KC * FB_AP;
        const bf16* Bb = Bs + (size_t)buf * FB_KC * FB_BP;
#pragma unroll
        for (int ks = 0; ks < FB_KC / 32; ++ks) {
            Raw8<bf16> fa[4], fb[4];
            const bf16* a0 = Ab + (size_t)(32 * ks + trow) * FB_AP + wr0 + tcol;
            const bf16* b0 = Bb + (size_t)(32 * ks + trow) * FB_BP + wc0 + tcol;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint2 lo = lds_tr4(a0 + 16 * i), hi = lds_tr4(a0 + 4 * FB_AP + 16 * i);
                fa[i].w[0] = lo.x; fa[i].w[1] = lo.y; fa[i].w[2] = hi.x; fa[i].w[3] = hi.y;
                const uint2 lb = lds_tr4(b0 + 16 * i), hb = lds_tr4(b0 + 4 * FB_BP + 16 * i);
                fb[i].w[0] = lb.x; fb[i].w[1] = lb.y; fb[i].w[2] = hb.x; fb[i].w[3] = hb.y;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) raw_mma(fa[i], fb[j], acc[i][j]);
        }
        commit(cur ^ 1, cur ^ 1);
        __syncthreads();
    };
    // (pairs with both calls unconditional: the register sets' states agree
    // at the top of every iteration)
    int ch = 0;
    for (; ch + 1 < nch; ch += 2) {
        chunk(ch, 0);
        chunk(ch + 1, 1);
    }
    if (ch < nch) chunk(ch, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int n = n0 + wc0 + 16 * j + (lane & 15);
        if (n >= G) continue;
        const float bn = a.bias[n];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + wr0 + 16 * i + acc_row(lane, r);
                if (row < B) a.Gx[((size_t)t * B + row) * G + n] = a.s * acc[i][j][r] + bn;
            }
    }
}

// ---------------------------------------------------------------------------
// Output-sparse input gradient for large batches (Eq. 10), summed over the
// directions:
//   dX_t[:, keep_t[j]] = s * sum_d DA_{d,t} W_d[keep_t[j], :]^T
// grid (8 * ceil(T/8) * ceil(K/128), 1, ceil(B/256)), 512 threads: workgroup i
// runs on XCD i % 8, which takes the steps t = i % 8 + 8j with all their
// column tiles, so DA_t is fetched into one XCD's L2 once.  A workgroup
// computes 256 rows x the 128 kept columns at keep-list positions 128*x ..
// (and, with
// scatter, writes the zeros of the dropped columns at drop-list positions
// 128*x ..); wave w owns rows 64*(w/2) and columns 64*(w%2) (4 x 4 tiles of
// 16x16x32 MFMA).  The contraction over 4H runs in chunks of 64: the DA
// chunk (fragment-major in memory: the MFMA operand layout) is copied to LDS
// as 1 KB blocks, the 128 gathered W rows' 64-column pieces are staged as
// [128][64+8] rows, double buffered, with the loads issued two chunks
// ahead; every fragment is one 16-byte LDS read.
constexpr int DB_M = 256, DB_N = 128, DB_KC = 64, DB_BP = DB_KC + 8;
constexpr size_t DB_LDS = (size_t)2 * (DB_M * DB_KC + DB_N * DB_BP) * 2 + (size_t)DB_N * 4;

__global__ void __launch_bounds__(512) k_dx_big(DxArgs a) {
    extern __shared__ __align__(16) char smem[];
    bf16* As = (bf16*)smem;                                  // [2][2 chunks][16 tiles][64 lanes][8]
    bf16* Bs = As + 2 * DB_M * DB_KC;                        // [2][DB_N][DB_BP]
    int* kcol = (int*)(Bs + 2 * DB_N * DB_BP);               // [DB_N] W rows of the tile's columns
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int ntile = (a.K + DB_N - 1) / DB_N;
    const int xcd = blockIdx.x % 8, idx = blockIdx.x / 8;
    const int t = xcd + 8 * (idx / ntile), j0 = (idx % ntile) * DB_N, m0 = blockIdx.z * DB_M;
    if (t >= a.T) return;
    const int B = a.B, G = a.G;
    const bool failed = a.status && *a.status != 0;
    const int cnt = a.site.count[t];
    const int32_t* krow = a.site.keep + (size_t)t * a.site.kmax;
    const uint8_t* mrow = a.site.mask + (size_t)t * a.site.kmax;
    float* out = a.out + (size_t)t * B * a.ldo;
    if (a.scatter) {                           // the dropped columns of this tile's drop-list range
        const int dn = a.site.dcount[t];
        const int32_t* drow = a.site.drop + (size_t)t * a.site.kmax;
        for (int i = tid; i < DB_N * DB_M; i += 512) {
            const int jj = j0 + (i % DB_N), row = m0 + i / DB_N;
            if (jj < dn && row < B) out[(size_t)row * a.ldo + drow[jj]] = failed ? __builtin_nanf("") : 0.0f;
        }
    }
    if (j0 >= cnt) return;
    if (tid < DB_N) kcol[tid] = j0 + tid < cnt ? krow[j0 + tid] : -1;
    __syncthreads();
    const int mt0 = m0 / 16;                   // first 16-row tile of the workgroup
    const size_t das = (size_t)((G + 31) / 32) * a.mtiles * 512;
    const int wr0 = 64 * (w >> 1), wc0 = 64 * (w & 1);
    const int g8 = 8 * (lane >> 4), cl = lane & 15;
    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
    const int nch = (G + DB_KC - 1) / DB_KC;
    for (int d = 0; d < a.D; ++d) {
        const __amdgpu_buffer_rsrc_t dr = buf_rsrc((const bf16*)a.da[d] + (size_t)t * das, (uint32_t)(das * 2));
        const __amdgpu_buffer_rsrc_t wr = buf_rsrc(a.W[d], (uint32_t)((size_t)a.K * G * 2));
        // staging: A = 2 chunks x 16 tiles of 1 KB (4 pieces per thread),
        // B = 128 rows x 8 pieces of 16 bytes (2 per thread); chunk c goes
        // through register set c % 2, its loads issued two chunks ahead
        u32x4_t ra[2][4], rb[2][2];
        auto fetch = [&](int set, int c) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = tid + 512 * i, blk = q >> 6, l = q & 63;   // blk = chunk half * 16 + tile
                const int ck = 2 * c + (blk >> 4), mt = mt0 + (blk & 15);
                const bool ok = mt < a.mtiles && 32 * ck < G;
                ra[set][i] = __builtin_amdgcn_raw_buffer_load_b128(
                    dr, ok ? (uint32_t)(frag_lane_off(ck, mt, l, a.mtiles) * 2) : OOB_OFF, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int q = tid + 512 * i, r = q >> 3, pc = q & 7;
                const int k = kcol[r], g = DB_KC * c + 8 * pc;
                rb[set][i] = __builtin_amdgcn_raw_buffer_load_b128(
                    wr, (k >= 0 && g < G) ? (uint32_t)(((size_t)k * G + g) * 2) : OOB_OFF, 0, 0);
            }
        };
        auto commit = [&](int set, int buf) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = tid + 512 * i;
                *(u32x4_t*)(As + (size_t)buf * DB_M * DB_KC + (size_t)q * 8) = ra[set][i];
            }
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int q = tid + 512 * i, r = q >> 3, pc = q & 7;
                *(u32x4_t*)(Bs + ((size_t)buf * DB_N + r) * DB_BP + 8 * pc) = rb[set][i];
            }
        };
        fetch(0, 0);
        fetch(1, 1);
        __syncthreads();                       // (the previous direction's last chunk is read)
        commit(0, 0);
        __syncthreads();
        auto chunk = [&](int c, int cur) {
            fetch(cur, c + 2);                 // (past the end: zeros, unconditionally)
            __builtin_amdgcn_sched_barrier(0);
            const int buf = cur;
            const bf16* Ab = As + (size_t)buf * DB_M * DB_KC;
            const bf16* Bb = Bs + (size_t)buf * DB_N * DB_BP;
#pragma unroll
            for (int ks = 0; ks < DB_KC / 32; ++ks) {
                Raw8<bf16> fa[4], fb[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    raw_lds(fa[i], Ab + ((size_t)(ks * 16 + (wr0 >> 4) + i) * 64 + lane) * 8);
                    raw_lds(fb[i], Bb + (size_t)(wc0 + 16 * i + cl) * DB_BP + 32 * ks + g8);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) raw_mma(fa[i], fb[j], acc[i][j]);
            }
            commit(cur ^ 1, cur ^ 1);
            __syncthreads();
        };
        int c = 0;
        for (; c + 1 < nch; c += 2) {
            chunk(c, 0);
            chunk(c + 1, 1);
        }
        if (c < nch) chunk(c, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int jl = wc0 + 16 * j + cl, jj = j0 + jl;
        if (jj >= cnt) continue;
        const int kk = kcol[jl];                 // (a kept column: a valid row)
        const float sc = (a.dense && !mrow[kk]) ? 0.0f : a.s;
        const int oc = a.scatter ? kk : jj;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = m0 + wr0 + 16 * i + acc_row(lane, r);
                if (row < B) out[(size_t)row * a.ldo + oc] = failed ? __builtin_nanf("") : sc * acc[i][j][r];
            }
    }
}

void launch_fx_big(const FxArgs& a, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid((a.G + FB_N - 1) / FB_N, a.T, (a.B + FB_M - 1) / FB_M), blk(512);
    if (e0 && e1) hipExtLaunchKernelGGL(k_fx_big, grid, blk, (uint32_t)FB_LDS, st, e0, e1, 0, a);
    else k_fx_big<<<grid, blk, FB_LDS, st>>>(a);
}
void launch_dx_big(const DxArgs& a, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid(8 * ((a.T + 7) / 8) * ((a.K + DB_N - 1) / DB_N), 1, (a.B + DB_M - 1) / DB_M), blk(512);
    if (e0 && e1) hipExtLaunchKernelGGL(k_dx_big, grid, blk, (uint32_t)DB_LDS, st, e0, e1, 0, a);
    else k_dx_big<<<grid, blk, DB_LDS, st>>>(a);
}

size_t wgrad_big_lds() { return WL_LDS; }

// The large-batch weight gradient takes any batch (its loads run two
// 64-row groups ahead); it pays off from a few groups per step on.
bool wgrad_big_fits(int B) { return B >= 64; }

// Weight gradient for large batches as one GEMM per problem, Eq. 11 with
// every row multiplied by its mask byte (a dropped row contributes an exact
// zero; identity keep lists need no mask):
//   dW[k][n] = s * sum over (t, b) of m_t[k] act_t[b][k] da_t[b][n]
// The contraction runs over all T*B (step, batch) pairs, so each
// workgroup's accumulators stay in registers for the whole pass: no per-step
// read-modify-write of an LDS accumulator (the row-sparse kernel above pays
// one for every kept row at every step, and at 256 rows per step that,
// with its per-step chain, holds it to about 10% of MFMA peak).
// grid (8 x row blocks x ceil(column blocks / 8), 1, problems), 512 threads;
// workgroup = 128 rows x 256 columns; workgroup i runs on XCD i % 8, which
// takes the column blocks i % 8 + 8j with every row block, so an XCD's L2
// holds its columns' DA^T for all of its row blocks.  Wave w owns rows
// 64 (w / 4) .. +63 and columns 64 (w % 4) .. +63 of the tile (4 x 4 MFMA
// tiles).  The contraction goes in chunks of 32 batch rows of one step: the
// chunk's 128 activation rows and 256 DA^T columns are loaded once (one or
// two 16-byte pieces per thread), stored fragment-major in LDS and read by
// the waves that need them.  Loads run up to five chunks ahead (register
// ring), three stage buffers rotate (a chunk is staged two chunks before it
// is multiplied), and each wave reads the fragments of the next chunk from
// LDS while it multiplies the current one; one barrier per chunk.  The workgroups of the
// last row block also sum the bias gradient.
constexpr int WM_R = 128, WM_C = 256, WM_KC = 32, WM_RING = 3;
constexpr size_t WM_STAGE = (size_t)(WM_R + WM_C) * WM_KC * 2;    // one stage buffer: 24 KB
constexpr size_t WM_LDS = 3 * WM_STAGE;

__global__ void __launch_bounds__(512) k_wgrad_gemm(WgBatch bt) {
    extern __shared__ __align__(16) char smem[];
    const WgArgs& a = bt.p[blockIdx.z];
    const int nrb = (a.K + WM_R - 1) / WM_R, ncb = (a.G + WM_C - 1) / WM_C;
    const int xcd = blockIdx.x % 8, k8 = blockIdx.x / 8;
    const int rb = k8 % nrb, cb = xcd + 8 * (k8 / nrb);
    if (cb >= ncb) return;
    const int r0 = rb * WM_R, n0 = cb * WM_C;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = w >> 2, wc = w & 3;
    const bool dbw = a.db && rb == nrb - 1;
    if (bt.status && *bt.status != 0) {        // the step's recurrence timed out: NaN in every output
        const float nan = __builtin_nanf("");
        for (int i = tid; i < WM_R * WM_C; i += 512) {
            const int r = r0 + i / WM_C, n = n0 + i % WM_C;
            if (r < a.K && n < a.G) a.out[(size_t)r * a.G + n] = nan;
        }
        if (dbw)
            for (int n = n0 + tid; n < min(n0 + WM_C, a.G); n += 512) a.db[n] = nan;
        return;
    }
    const bool masked = a.dense || !a.full;    // rows times the mask byte
    const int nb = (a.B + WM_KC - 1) / WM_KC, nq = a.T * nb;
    const uint32_t abytes = (uint32_t)a.K * a.BP * 2, bbytes = (uint32_t)a.G * a.BP * 2;
    // staging pieces of this thread: activation row j, DA^T columns j and
    // j + 128, batch entries 8 q4 .. +7 of the chunk
    // (lane l of a wave takes fragment position l of a 16-row tile, so a
    // wave's LDS stores are one contiguous 1 KB block: no bank conflicts)
    const int j = (tid & 15) + 16 * (tid >> 6), q4 = (tid >> 4) & 3;
    const int frag = ((j & 15) + 16 * q4) * 16 + (j >> 4) * 1024;   // fragment-major offset in a 16-row tile
    const bool rok = r0 + j < a.K;
    auto act_rsrc = [&](int t) {
        const bf16* act = (a.actT_first && t == a.t_first) ? (const bf16*)a.actT_first
                                                           : (const bf16*)a.actT + (long)(t + a.shift) * a.tstride;
        return buf_rsrc(act, abytes);
    };
    // per-thread byte offsets of the pieces within a step's blocks (chunk 0);
    // chunk c of the step adds 64 c bytes (out-of-range offsets stay so)
    const uint32_t aoff = rok ? (uint32_t)((r0 + j) * a.BP + 8 * q4) * 2 : OOB_OFF;
    const uint32_t boff0 = n0 + j < a.G ? (uint32_t)((n0 + j) * a.BP + 8 * q4) * 2 : OOB_OFF;
    const uint32_t boff1 = n0 + 128 + j < a.G ? (uint32_t)((n0 + 128 + j) * a.BP + 8 * q4) * 2 : OOB_OFF;
    const uint32_t moff = masked && rok ? (uint32_t)(r0 + j) : OOB_OFF;
    const bool padb = (a.B & (WM_KC - 1)) != 0;   // the last chunk of a step holds padding rows
    auto dat_rsrc = [&](int t) { return buf_rsrc((const bf16*)a.daT + (size_t)t * a.G * a.BP, bbytes); };
    auto msk_rsrc = [&](int t) { return buf_rsrc(a.site.mask + (size_t)t * a.site.kmax, (uint32_t)a.site.kmax); };
    // the next chunk to load (chunks go out in order): its step, its index
    // in the step, its index, and the step's resources; past the last chunk
    // the last one is loaded again
    int it = 0, ic = 0, iq = 0;
    __amdgpu_buffer_rsrc_t ar = act_rsrc(0), br = dat_rsrc(0), mr = msk_rsrc(0);
    u32x4_t ra[WM_RING], rb0[WM_RING], rb1[WM_RING];
    int mk[WM_RING], bq[WM_RING];
    auto issue = [&](int sl) {
        const uint32_t co = 64u * ic;
        bq[sl] = WM_KC * ic + 8 * q4;
        ra[sl] = __builtin_amdgcn_raw_buffer_load_b128(ar, aoff + co, 0, 0);
        rb0[sl] = __builtin_amdgcn_raw_buffer_load_b128(br, boff0 + co, 0, 0);
        rb1[sl] = __builtin_amdgcn_raw_buffer_load_b128(br, boff1 + co, 0, 0);
        // (always issued, past the resource when not masked or past the rows)
        mk[sl] = (int)__builtin_amdgcn_raw_buffer_load_b8(mr, moff, 0, 0);
        if (iq + 1 < nq) {
            ++iq;
            if (++ic == nb) {
                ic = 0;
                ++it;
                ar = act_rsrc(it);
                br = dat_rsrc(it);
                mr = msk_rsrc(it);
            }
        }
    };
    auto stage = [&](int buf, int sl) {
        uint32_t pm[4] = {~0u, ~0u, ~0u, ~0u};
        if (padb) pad_mask<bf16>(bq[sl], a.B, pm);
        char* sb = smem + buf * WM_STAGE;
        const bool keep = !masked || mk[sl] != 0;
        const uint4 va = keep ? make_uint4(ra[sl][0] & pm[0], ra[sl][1] & pm[1], ra[sl][2] & pm[2], ra[sl][3] & pm[3])
                              : make_uint4(0u, 0u, 0u, 0u);
        *(uint4*)(sb + frag) = va;
        *(uint4*)(sb + WM_R * WM_KC * 2 + frag) =
            make_uint4(rb0[sl][0] & pm[0], rb0[sl][1] & pm[1], rb0[sl][2] & pm[2], rb0[sl][3] & pm[3]);
        *(uint4*)(sb + WM_R * WM_KC * 2 + 8 * 1024 + frag) =
            make_uint4(rb1[sl][0] & pm[0], rb1[sl][1] & pm[1], rb1[sl][2] & pm[2], rb1[sl][3] & pm[3]);
    };
    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[i][c] = f32x4_t{0, 0, 0, 0};
    // the bias gradient (the last row block's waves 0-3): each DA^T fragment
    // times a fragment of ones, i.e. its column sums over the chunk's batch
    // entries, on the matrix cores (unpacking and adding the bf16 pairs took
    // 64 vector instructions per chunk, and those workgroups set the
    // kernel's time)
    f32x4_t dbacc[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) dbacc[c] = f32x4_t{0, 0, 0, 0};
    Raw8<bf16> ones;
#pragma unroll
    for (int q = 0; q < Raw8<bf16>::NW; ++q) ones.w[q] = 0x3f803f80u;     // bf16 1.0, twice
    // fragments of two chunks in registers: those of chunk q+1 are read
    // from LDS while chunk q is multiplied
    Raw8<bf16> fa[2][4], fb[2][4];
    auto frags = [&](int buf, int fs) {
        const char* sb = smem + buf * WM_STAGE;
#pragma unroll
        for (int c = 0; c < 4; ++c) raw_lds(fb[fs][c], (const bf16*)(sb + WM_R * WM_KC * 2 + (4 * wc + c) * 1024 + lane * 16));
#pragma unroll
        for (int i = 0; i < 4; ++i) raw_lds(fa[fs][i], (const bf16*)(sb + (4 * wr + i) * 1024 + lane * 16));
    };
    auto multiply = [&](int fs) {
        if (dbw && wr == 0)
#pragma unroll
            for (int c = 0; c < 4; ++c) raw_mma(fb[fs][c], ones, dbacc[c]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < 4; ++c) raw_mma(fb[fs][c], fa[fs][i], acc[i][c]);
    };
    // chunk q: stage q+2 (its loads went out two chunks earlier) into the
    // third buffer, read the fragments of q+1, multiply q, then the slot of
    // q+2 takes the loads of q+2+WM_RING
    // (sl = q % WM_RING and fs = q % 2, passed as constants of the unrolled loop)
    auto iter = [&](int q, int sl, int fs) {
        stage((q + 2) % 3, (sl + 2) % WM_RING);
        frags((q + 1) % 3, fs ^ 1);
        if (q < nq) multiply(fs);
        issue((sl + 2) % WM_RING);               // (chunk q + 2 + WM_RING)
        __syncthreads();
    };
#pragma unroll
    for (int i = 0; i < WM_RING; ++i) issue(i);
    stage(0, 0);
    stage(1, 1);
    issue(0);
    issue(1);
    __syncthreads();
    frags(0, 0);
    for (int q = 0; q < nq; q += 2 * WM_RING) {
#pragma unroll
        for (int i = 0; i < 2 * WM_RING; ++i) iter(q + i, i % WM_RING, i & 1);
    }
    // (transposed products) output r of this lane is gradient column
    // 4*(lane/16)+r of the column tile, in the lane's own row
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = r0 + 64 * wr + 16 * i + (lane & 15);
        if (row >= a.K) continue;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int nq4 = n0 + 64 * wc + 16 * c + 4 * (lane >> 4);
            float* o = a.out + (size_t)row * a.G + nq4;
            if (nq4 + 3 < a.G) {
                *(float4*)o = make_float4(a.s * acc[i][c][0], a.s * acc[i][c][1], a.s * acc[i][c][2], a.s * acc[i][c][3]);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (nq4 + r < a.G) o[r] = a.s * acc[i][c][r];
            }
        }
    }
    if (dbw && wr == 0 && (lane & 15) == 0) {  // (every output column holds the same sums) output r of
#pragma unroll                                 // lane 16j is the sum of tile column 4j+r
        for (int c = 0; c < 4; ++c)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int n = n0 + 64 * wc + 16 * c + 4 * (lane >> 4) + r;
                if (n < a.G) a.db[n] = dbacc[c][r];
            }
    }
}

void launch_wgrad_gemm(const WgBatch& b, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    int nx = 0;                                // 8 x (row blocks) x ceil(column blocks / 8)
    for (int i = 0; i < b.np; ++i)
        nx = std::max(nx, 8 * ((b.p[i].K + WM_R - 1) / WM_R) * (((b.p[i].G + WM_C - 1) / WM_C + 7) / 8));
    const dim3 grid(nx, 1, b.np), blk(512);
    if (e0 && e1) hipExtLaunchKernelGGL(k_wgrad_gemm, grid, blk, (uint32_t)WM_LDS, st, e0, e1, 0, b);
    else k_wgrad_gemm<<<grid, blk, WM_LDS, st>>>(b);
}

void launch_wgrad_big(const WgBatch& b, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    int nx = 0;                                // 8 x (row slices) x ceil(column blocks / 8)
    for (int i = 0; i < b.np; ++i)
        nx = std::max(nx, 8 * ((b.p[i].K + WL_R - 1) / WL_R) * (((b.p[i].G + WL_C - 1) / WL_C + 7) / 8));
    const dim3 grid(nx, 1, b.np), blk(512);
    if (e0 && e1) hipExtLaunchKernelGGL(k_wgrad_big, grid, blk, (uint32_t)wgrad_big_lds(), st, e0, e1, 0, b);
    else k_wgrad_big<<<grid, blk, wgrad_big_lds(), st>>>(b);
}

int setup_big_attributes() {
    bool ok = hipFuncSetAttribute((const void*)k_wgrad_big, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)wgrad_big_lds()) == hipSuccess;
    ok = hipFuncSetAttribute((const void*)k_fx_big, hipFuncAttributeMaxDynamicSharedMemorySize, (int)FB_LDS) ==
             hipSuccess && ok;
    ok = hipFuncSetAttribute((const void*)k_dx_big, hipFuncAttributeMaxDynamicSharedMemorySize, (int)DB_LDS) ==
             hipSuccess && ok;
    ok = hipFuncSetAttribute((const void*)k_wgrad_gemm, hipFuncAttributeMaxDynamicSharedMemorySize, (int)WM_LDS) ==
             hipSuccess && ok;
    return ok ? 0 : -1;
}

}  // namespace lsd
