// Products of the step at large batches (gfx950, bf16): the weight
// gradients (Eq. 11) as a contraction over the batch on 32x32x16 MFMA tiles.
// At a batch of a few hundred rows the contraction is long enough for the
// products to be bound by MFMA and cache bandwidth, so these kernels keep
// their accumulators in registers over the batch and feed the MFMAs from
// loads issued several contraction steps ahead, where the small-batch
// kernels (one contraction chunk per step) are bound by per-step latency.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>

#include "device.h"
#include "kernels.h"
#include "../../include/lstm_sd.h"

namespace lsd {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Operand fragment of v_mfma_f32_32x32x16_bf16: lane l holds row (A) or
// column (B) l % 32 and contraction elements 8*(l/32) .. 8*(l/32)+7 of a
// 16-long step; result element i of lane l is row 8*(i/4) + 4*(l/32) + i%4,
// column l % 32.
__device__ __forceinline__ int acc32_row(int lane, int i) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

// ---------------------------------------------------------------------------
// Weight gradient for large batches, Eq. 11:
//   dW[k][n] = s * sum_t sum_{b} act_t[b][k] da_t[b][n]   over the steps t
// at which row k is kept (row-sparse), or every step with the mask as a
// multiplier (the dense comparison mode); rows never kept are 0.
// grid (row slices of 128 x column blocks of 128, 1, problems), 512 threads.
// Per step the workgroup lists the kept rows of its slice (a ballot over the
// mask bytes), wave w multiplies the kept-row tiles rp, rp+2 (rp = w/4) of
// 32 rows with column tile w%4 of 32 columns over the batch (16-long MFMA
// steps, operands loaded two 64-row groups ahead across step boundaries), and adds
// the tiles into the slice's rows of an LDS accumulator (kept rows of one
// step are distinct; absent tile rows go to a spare row).  Slice 0 also sums
// the bias gradient.  One launch covers every problem of a pass.
constexpr int WB_R = 128, WB_C = 128, WB_LDC = WB_C + 4;

__global__ void __launch_bounds__(512) k_wgrad_big(WgBatch bt) {
    extern __shared__ __align__(16) char smem[];
    const WgArgs& a = bt.p[blockIdx.z];
    const int nrs = (a.K + WB_R - 1) / WB_R, ncb = (a.G + WB_C - 1) / WB_C;
    // workgroup i runs on XCD i % 8: each XCD takes the column blocks
    // x, x+8, ... with every row slice, so one XCD's L2 holds its columns'
    // DA^T of a step once for all of its slices (column blocks across XCDs
    // would make every XCD read all of DA^T)
    const int xcd = blockIdx.x % 8, k8 = blockIdx.x / 8;
    const int rs = k8 % nrs, cb = xcd + 8 * (k8 / nrs);
    if (cb >= ncb) return;
    const int r0 = rs * WB_R, nrow = min(WB_R, a.K - r0), n0 = cb * WB_C;
    float* acc_lds = (float*)smem;                                // [WB_R + 1][WB_LDC]
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    int* rowlist = (int*)(smem + (size_t)(WB_R + 1) * WB_LDC * 4) + w * 2 * WB_R;   // [2][WB_R] per wave
    const int rp = w >> 2, ct = w & 3;
    const int B = a.B, G = a.G, T_ = a.T;
    const bool failed = bt.status && *bt.status != 0;
    for (int i = tid; i < (WB_R + 1) * WB_LDC; i += 512) acc_lds[i] = 0.0f;
    __syncthreads();

    const int ncol = n0 + 32 * ct + (lane & 31);                  // this lane's B column
    const uint32_t boff = (uint32_t)(min(ncol, G - 1) * a.BP + 32 * (lane >> 5)) * 2;   // this lane's DA^T row and half
    const bool dbw = a.db && rs == 0 && rp == 0;                  // sums the bias gradient
    float dbacc = 0.0f;

    // mask bytes of the slice's rows r0 + lane and r0 + 64 + lane at step t
    // (clamped, valid addresses; loaded a step before they are used)
    auto mask_load = [&](int t, uint32_t& k0, uint32_t& k1) {
        const uint8_t* mrow = a.site.mask + (size_t)min(t, T_ - 1) * a.site.kmax + r0;
        k0 = mrow[min(lane, nrow - 1)];
        k1 = mrow[min(lane + 64, nrow - 1)];
    };
    // the rows of a step from its mask bytes: kept rows of the slice in
    // ascending order (compact mode) or every row (dense mode); returns the
    // count
    auto build = [&](uint32_t mk0, uint32_t mk1, int* rl) -> int {
        const bool k0 = lane < nrow && mk0 != 0;
        const bool k1 = lane + 64 < nrow && mk1 != 0;
        if (a.dense) {
            rl[lane] = r0 + min(lane, nrow - 1);
            rl[lane + 64] = r0 + min(lane + 64, nrow - 1);
            return nrow;
        }
        const uint64_t b0 = __builtin_amdgcn_ballot_w64(k0), b1 = __builtin_amdgcn_ballot_w64(k1);
        const int c0 = __popcll(b0);
        const int i0 = __builtin_amdgcn_mbcnt_hi((uint32_t)(b0 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b0, 0));
        const int i1 = c0 + __builtin_amdgcn_mbcnt_hi((uint32_t)(b1 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b1, 0));
        if (k0) rl[i0] = r0 + lane;
        if (k1) rl[i1] = r0 + 64 + lane;
        return c0 + __popcll(b1);
    };
    auto act_ptr = [&](int t) {
        return (a.actT_first && t == a.t_first) ? (const bf16*)a.actT_first
                                                : (const bf16*)a.actT + (long)(t + a.shift) * a.tstride;
    };

    // The contraction over the batch runs in groups of 64 batch rows (one
    // 128-byte line of an operand row): MFMA step j (0..3) of group g takes,
    // on lane half h, the 8 batch rows 64g + 32h + 8j (the order inside a
    // group only has to agree between the two operands), so the four steps'
    // loads of a lane read 64 contiguous bytes and a row's line is used up
    // by one group.  Flattened pipeline over q = t * ng + g, two groups of
    // operands in flight: slot q & 1 holds group q, and receives q + 2 (of
    // step t or t+1) once q is multiplied.  Loads are unconditional (clamped
    // q; rows of absent tiles point at one row), so the compiler keeps exact
    // wait counts.  The row lists of two steps are kept: cur (step t) and nxt
    // (t+1); the list of t+2 is built once t is done.
    struct Rows { int n; uint32_t ao[2]; uint32_t dm[2]; };     // ao: A row and lane-half byte offsets
    auto prep = [&](int t, uint32_t mk0, uint32_t mk1, Rows& R) {
        int* rl = rowlist + (t & 1) * WB_R;
        R.n = __builtin_amdgcn_readfirstlane(build(mk0, mk1, rl));
        // (wave-local LDS: the writes above come before the reads below in program order)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int j = 32 * (rp + 2 * i) + (lane & 31);
            const int r = j < R.n ? rl[j] : r0;
            R.ao[i] = (uint32_t)r * a.BP * 2 + (uint32_t)(32 * (lane >> 5)) * 2;
            // dense mode: the mask byte of row r0 + j sits in lane j % 64
            const uint32_t mj = (uint32_t)__shfl((int)(j < 64 ? mk0 : mk1), j & 63);
            R.dm[i] = a.dense ? (uint32_t)(mj != 0) : 1u;
        }
    };
    const int ng = (B + 63) / 64;                                 // 64-row groups of the batch
    u32x4_t fa[2][4][2], fb[2][4];
    auto issue = [&](int q, const Rows& R, u32x4_t (&fa_)[4][2], u32x4_t (&fb_)[4]) {
        const int t = min(q / ng, T_ - 1), g = q % ng;
        const __amdgpu_buffer_rsrc_t ar = buf_rsrc(act_ptr(t), (uint32_t)a.K * a.BP * 2);
        const __amdgpu_buffer_rsrc_t br = buf_rsrc((const bf16*)a.daT + (size_t)t * G * a.BP, (uint32_t)G * a.BP * 2);
        const uint32_t gb = (uint32_t)(128 * g);                  // the group's bytes within a row
        const uint32_t bo = boff + gb, ao0 = R.ao[0] + gb, ao1 = R.ao[1] + gb;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            fa_[j][0] = __builtin_amdgcn_raw_buffer_load_b128(ar, ao0 + 16 * j, 0, 0);
            fa_[j][1] = __builtin_amdgcn_raw_buffer_load_b128(ar, ao1 + 16 * j, 0, 0);
            fb_[j] = __builtin_amdgcn_raw_buffer_load_b128(br, bo + 16 * j, 0, 0);
        }
    };

    f32x16_t acc[2];
    Rows cur, nxt;
    uint32_t mk0, mk1;                                            // mask bytes of step t+2, in flight
    mask_load(0, mk0, mk1);
    prep(0, mk0, mk1, cur);
    mask_load(1, mk0, mk1);
    prep(min(1, T_ - 1), mk0, mk1, nxt);
    mask_load(2, mk0, mk1);
    issue(0, cur, fa[0], fb[0]);
    issue(1, ng > 1 ? cur : nxt, fa[1], fb[1]);
    for (int q0 = 0; q0 < T_ * ng; q0 += 2) {
#pragma unroll
        for (int sl = 0; sl < 2; ++sl) {
            const int q = q0 + sl;
            if (q >= T_ * ng) break;
            const int t = q / ng, g = q % ng;
            if (g == 0) {
#pragma unroll
                for (int i = 0; i < 2; ++i) acc[i] = f32x16_t{};
            }
            const bool act0 = 32 * rp < cur.n, act1 = 32 * (rp + 2) < cur.n;   // (uniform) tiles with kept rows
            const bool pad = 64 * (g + 1) > B;                    // batch rows past B in this group
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                u32x4_t b = fb[sl][j];
                u32x4_t av0 = fa[sl][j][0], av1 = fa[sl][j][1];
                if (pad) {
                    uint32_t m[4];
                    pad_mask<bf16>(64 * g + 32 * (lane >> 5) + 8 * j, B, m);
#pragma unroll
                    for (int e = 0; e < 4; ++e) { b[e] &= m[e]; av0[e] &= m[e]; av1[e] &= m[e]; }
                }
                if (dbw && ncol < G) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) dbacc += __uint_as_float(b[e] << 16) + __uint_as_float(b[e] & 0xffff0000u);
                }
                const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, b);
                if (act0) {
                    const u32x4_t x = cur.dm[0] ? av0 : u32x4_t{0, 0, 0, 0};   // dense mode: a dropped row
                    acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, x), bv, acc[0], 0, 0, 0);
                }
                if (act1) {
                    const u32x4_t x = cur.dm[1] ? av1 : u32x4_t{0, 0, 0, 0};
                    acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, x), bv, acc[1], 0, 0, 0);
                }
            }
            const bool last = g == ng - 1;
            // group q + 2 belongs to step t (cur) or t+1 (nxt); q + 2 of step
            // t+2 only when ng == 1, in which case it is issued after the
            // lists advance below
            if (ng > 1) issue(q + 2, (q + 2) / ng == t ? cur : nxt, fa[sl], fb[sl]);
            if (last) {
                // the tiles of step t into their rows of the accumulator.  A
                // row's compacted position, and so the wave that adds it,
                // changes from step to step: every wave's additions of step
                // t-1 are complete before any of step t begins.  Within a
                // step the rows of the tiles are distinct (absent ones go to
                // the spare row), so all old values are read before any is
                // written.
                __syncthreads();
                const int* rl = rowlist + (t & 1) * WB_R;
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    if (!(i == 0 ? act0 : act1)) continue;
                    const int tb = 32 * (rp + 2 * i);
                    float* dst[16];
                    float old[16];
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int jj = tb + acc32_row(lane, e);
                        const int r = jj < cur.n ? rl[min(jj, WB_R - 1)] - r0 : WB_R;
                        dst[e] = acc_lds + r * WB_LDC + 32 * ct + (lane & 31);
                    }
#pragma unroll
                    for (int e = 0; e < 16; ++e) old[e] = *dst[e];
#pragma unroll
                    for (int e = 0; e < 16; ++e) *dst[e] = old[e] + a.s * acc[i][e];
                }
                cur = nxt;
                if (t + 2 < T_) prep(t + 2, mk0, mk1, nxt);       // (the list of t is no longer read)
                mask_load(t + 3, mk0, mk1);
            }
            if (ng == 1) issue(q + 2, nxt, fa[sl], fb[sl]);       // (step t+2: nxt after the advance)
        }
    }
    __syncthreads();
    const float nan = __builtin_nanf("");
    for (int i = tid; i < nrow * WB_C; i += 512) {
        const int r = i / WB_C, c = i % WB_C;
        if (n0 + c < G) a.out[(size_t)(r0 + r) * G + n0 + c] = failed ? nan : acc_lds[r * WB_LDC + c];
    }
    if (dbw) {
        dbacc += __shfl_xor(dbacc, 32);
        if (lane < 32 && ncol < G) a.db[ncol] = failed ? nan : dbacc;
    }
}

size_t wgrad_big_lds() { return (size_t)(WB_R + 1) * WB_LDC * 4 + (size_t)8 * 2 * WB_R * 4; }

// The large-batch weight gradient takes any batch (its loads run two
// 64-row groups ahead); it pays off from a few groups per step on.
bool wgrad_big_fits(int B) { return B >= 64; }

void launch_wgrad_big(const WgBatch& b, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    int nx = 0;                                // 8 x (row slices) x ceil(column blocks / 8)
    for (int i = 0; i < b.np; ++i)
        nx = std::max(nx, 8 * ((b.p[i].K + WB_R - 1) / WB_R) * (((b.p[i].G + WB_C - 1) / WB_C + 7) / 8));
    const dim3 grid(nx, 1, b.np), blk(512);
    if (e0 && e1) hipExtLaunchKernelGGL(k_wgrad_big, grid, blk, (uint32_t)wgrad_big_lds(), st, e0, e1, 0, b);
    else k_wgrad_big<<<grid, blk, wgrad_big_lds(), st>>>(b);
}

int setup_big_attributes() {
    return hipFuncSetAttribute((const void*)k_wgrad_big, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)wgrad_big_lds()) == hipSuccess ? 0 : -1;
}

}  // namespace lsd
