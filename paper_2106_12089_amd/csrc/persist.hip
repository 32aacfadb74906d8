// Persistent recurrent kernels (gfx950): one launch runs every
// time step of a layer.  Each workgroup keeps its slice of the recurrent
// weight U in LDS and its part of the cell state in registers for the whole
// sequence; the workgroups meet at a grid barrier once per step.
//
// The producer of h_t knows the next step's keep list (all masks are drawn
// before the forward pass), so it writes h_t already compacted by that list
// ("compaction at the producer"): the consumer reads its MFMA A fragments as
// contiguous 16-byte loads and never touches a dropped column.
#include <hip/hip_runtime.h>

#include <stdlib.h>

#include <mutex>
#include <vector>

#include "device.h"
#include "kernels.h"
#include "sync.h"
#include "../../include/lstm_sd.h"

namespace lsd {

// ---------------------------------------------------------------------------
// Persistent forward recurrence (Eq. 1-6).  A launch runs every step of its
// slots: the two directions of one layer, or every layer of a
// unidirectional stack together with one input-product worker per layer
// above the first.  The worker of layer l forms gx_t = s_nr * x~_t W + b
// (Eq. 1-4, input part) as soon as layer l-1 has published x_t, and layer l
// reads it like the first layer reads the input product of the separate
// pass; so the recurrence of every layer only waits for its own barrier.
// Workgroup w -> (slot, unit tile, row group).  A unit tile is 4*NT hidden
// units = NT 16-column MFMA tiles (the four gates of 4 units each); a row
// group is MG batch rows.  512 threads = 8 waves; each contraction over kept
// neurons is split over the waves (each wave issues all of its exchange
// loads before its first MFMA) and reduced in LDS.
// Dynamic LDS: the weight slice, U for a layer, W for a worker, with HP =
// fwd_hp(H) (or KP) rows: rows of the weight rounded up to 32, plus 8, zero
// past the end.  bf16 slices are K-major, [HP][16*NT + 4]: the B fragment of
// a 16-column tile over 32 kept neurons is two transposing 8-byte LDS reads
// per lane, whose addresses are the kept rows of the keep list, so a
// gathered fragment costs what a contiguous one does.  f32 slices are
// column-major, [16*NT][HP], a fragment one 32-byte read (identity keep
// list) or 8 gathered elements.  Then keep lists [H+32] and [kin_max+32]
// (int16) and the reduction area [8][MG][16*NT] (float).
constexpr int PF_NW = 8;
__host__ __device__ constexpr int fwd_ncp(int NT) { return 16 * NT + 4; }

template <typename T, int NT, int MG>
__global__ void __launch_bounds__(512) k_fwd_persist(PFwdArgs a) {
    constexpr int UPW = 4 * NT, MT = MG / 16, NW = PF_NW, NC = 16 * NT;
    constexpr int NTH = 64 * NW;
    constexpr int PPT = (MG * UPW + NTH - 1) / NTH;
    constexpr int MAXC = MT <= 2 ? 3 : 2;       // chunks per wave per round (registers)
    constexpr bool KM = sizeof(T) == 2;          // K-major weight slices (transposing reads)
    constexpr int NCP = fwd_ncp(NT);             // their row pitch (elements)
    extern __shared__ __align__(16) char smem[];
    const int H = a.H, G = 4 * H, B = a.B, T_ = a.T;
    const int HP = fwd_hp(H), KP = a.KP;
    T* Ut = (T*)smem;                             // a layer's U slice
    T* Wt = (T*)(smem + a.wofs);                  // the W slice (a worker's: in place of U)
    int16_t* kidx = (int16_t*)(smem + a.kofs);
    int16_t* kidx_x = kidx + (((H + 32) + 7) & ~7);
    float* red = (float*)((char*)kidx_x + (KP ? (((size_t)(a.kin_max + 32) * 2 + 15) & ~(size_t)15) : 0));

    const int nslot = a.ntiles * a.mgroups;
    const int d = blockIdx.x / nslot, rem = blockIdx.x % nslot;
    const int tile = rem / a.mgroups, mg = rem % a.mgroups;
    const PFwdDir& D = a.d[d];
    const int u0 = tile * UPW, m0 = mg * MG;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int g8 = 8 * (lane >> 4);
    unsigned* bar = slot_bar(a.bar, d);
    // the slot this one depends on: a slot forming an input product, the
    // layer below (step s needs its counter at (s+2)*nslot: it also arrives
    // once before its first step); a layer fed by a worker, that worker
    // ((s+1)*nslot)
    unsigned* bar_dep = D.dep >= 0 ? slot_bar(a.bar, D.dep) : nullptr;
    __shared__ unsigned dep_seen;                 // steps of that slot last seen complete
    unsigned seen_dep = 0;                        // its copy in every thread
    const bool worker = D.role == 1;
    const bool has_x = D.Win != nullptr;          // forms an input product (a worker, or a layer itself)
    const bool fed = !has_x && D.dep >= 0;        // a layer reading its worker's input product
    const int kin = D.kin;

    // U slice (or W slice) -> LDS: column c = nt*16 + cu*4 + g of the slice
    // is column g*H + u0 + 4nt + cu of the weight (the four gates of a unit
    // side by side, so the reduction reads them as one 16-byte piece).
    // Each thread issues its loads
    // in batches of LB from clamped (valid) addresses before storing any: a
    // loop of load-then-store waits a full memory latency per element.
    {
        constexpr int LB = 16;
        auto load_slice = [&](const T* Wm, int rows, int krows, T* dst, int pitch) {
            const int total = pitch * NC;
            for (int i0 = tid; i0 < total; i0 += NTH * LB) {
                T v[LB];
#pragma unroll
                for (int j = 0; j < LB; ++j) {
                    const int i = min(i0 + NTH * j, total - 1);
                    const int k = i / NC, c = i % NC;
                    const int u = u0 + 4 * (c >> 4) + ((c & 15) >> 2);
                    v[j] = Wm[(size_t)min(k, krows - 1) * G + (c & 3) * H + min(u, H - 1)];
                }
#pragma unroll
                for (int j = 0; j < LB; ++j) {
                    const int i = i0 + NTH * j;
                    if (i < total) {
                        const int k = i / NC, c = i % NC;
                        const int u = u0 + 4 * (c >> 4) + ((c & 15) >> 2);
                        dst[KM ? k * NCP + c : c * pitch + k] = (u < H && k < rows) ? v[j] : zero_val<T>();
                    }
                }
            }
        };
        if (!worker) load_slice((const T*)D.U, H, H, Ut, HP);
        if (has_x) load_slice((const T*)D.Win, kin, kin, Wt, KP);
        // keep-list entries past a step's count are read as rows (their A
        // side is zero): they always hold a valid row index
        for (int i = tid; i < H + 32; i += NTH) kidx[i] = 0;
        if (KP)
            for (int i = tid; i < a.kin_max + 32; i += NTH) kidx_x[i] = 0;
    }
    // register state of this thread's (row, unit) pairs
    float creg[PPT], hreg[PPT], biasr[PPT][4];
    int pb[PPT], pu[PPT];
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        const int p = tid + NTH * q;
        const int rr = p / UPW, uu = p % UPW;
        pb[q] = (p < MG * UPW) ? m0 + rr : B;
        pu[q] = u0 + uu;
        const bool ok = pb[q] < B && pu[q] < H && !worker;
        creg[q] = ok ? D.c0[(size_t)pb[q] * H + pu[q]] : 0.f;
        hreg[q] = ok ? to_f32<T>(((const T*)D.h0)[(size_t)pb[q] * H + pu[q]]) : 0.f;
#pragma unroll
        for (int g = 0; g < 4; ++g) biasr[q][g] = has_x ? D.bias[g * H + min(pu[q], H - 1)] : 0.f;
    }
    // per-step inputs that do not depend on the recurrence, loaded one step
    // ahead from clamped (valid) addresses without branches; pointwise uses
    // them only for valid (row, unit) pairs
    float gxr[PPT][4];
    int pn[PPT], mnr[PPT], lenr[PPT], pup[PPT], mup[PPT];
    int cnt = 0, cnt_next = 0, cnt_x = 0, cnt_x_next = 0;
    constexpr int KPT = (LSTM_SD_MAX_K + NTH - 1) / NTH;   // keep-list entries per thread
    int kreg[KPT], kreg_x[KPT];
    auto step_t = [&](int s) { return D.dir == 0 ? s : T_ - 1 - s; };
    auto load_gx = [&](int t) {                   // input product and bias of step t
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int bc = min(pb[q], B - 1), uc = min(pu[q], H - 1);
            const float* p = D.gx + ((size_t)t * B + bc) * G + uc;
#pragma unroll
            for (int g = 0; g < 4; ++g)         // (a fed layer's come from its worker in this launch)
                gxr[q][g] = fed ? xload1(p + g * H) : p[g * H];
        }
    };
    auto prefetch = [&](int s) {                  // s may be T_ (after the last step): clamped
        const int sc = min(s, T_ - 1);
        const int t = step_t(sc);
        const bool has_next = sc + 1 < T_;
        const int tn = has_next ? step_t(sc + 1) : t;
        // (counts made wave-uniform: the buffer resources sized by them are
        // then scalar; a count from a vector load wrapped every exchange
        // load in a loop over the resource's distinct values)
        cnt_next = __builtin_amdgcn_readfirstlane(D.rh.count[t]);
        const int32_t* krow = D.rh.keep + (size_t)t * D.rh.kmax;
#pragma unroll
        for (int i = 0; i < KPT; ++i) kreg[i] = krow[min(tid + NTH * i, D.rh.kmax - 1)];
        if (has_x) {
            cnt_x_next = __builtin_amdgcn_readfirstlane(D.nr.count[t]);
            const int32_t* kx = D.nr.keep + (size_t)t * D.nr.kmax;
#pragma unroll
            for (int i = 0; i < KPT; ++i) kreg_x[i] = kx[min(tid + NTH * i, D.nr.kmax - 1)];
        }
        if (!has_x && !fed) load_gx(t);           // (a fed layer loads it once its worker has published it)
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int bc = min(pb[q], B - 1), uc = min(pu[q], H - 1);
            pn[q] = has_next ? D.rh.pos[(size_t)tn * D.rh.kmax + uc] : -1;
            mnr[q] = D.rh.mask[(size_t)tn * D.rh.kmax + uc];
            lenr[q] = a.lengths ? a.lengths[bc] : T_;
            if (D.xout) {
                pup[q] = D.nr_up.pos[(size_t)t * D.nr_up.kmax + uc];
                mup[q] = D.nr_up.mask[(size_t)t * D.nr_up.kmax + uc];
            }
        }
    };
    auto is_valid = [&](int q, int t) { return pb[q] < B && pu[q] < H && t < lenr[q]; };

    // the keep lists of the coming step, from registers to LDS
    auto commit_kidx = [&]() {
        cnt = cnt_next;
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            const int j = tid + NTH * i;
            if (j < cnt) kidx[j] = (int16_t)kreg[i];
        }
    };
    auto commit_kidx_x = [&]() {
        cnt_x = cnt_x_next;
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            const int j = tid + NTH * i;
            if (j < cnt_x) kidx_x[j] = (int16_t)kreg_x[i];
        }
    };

    // acc += (compacted A from the exchange) x (weight slice rows of the keep
    // list), in rounds of NW*MAXC 32-neuron chunks.  src holds one step's
    // fragment-major slot of slot_elems elements, Bt the transposed weight
    // slice of pitch bp, kfull the contraction length when nothing is
    // dropped.  issue() loads the A fragments of round c0 (chunks past the
    // slot, and lanes of rows past B, read as 0 without moving data);
    // compute() multiplies every chunk slot of the
    // round (slots past the keep count have a zeroed A side and read B rows at
    // offset 0: no branch lets the compiler sink the loads into the products).
    auto issue = [&](const T* src, size_t slot_elems, int n, int c0, Raw8<T> (&fa)[MAXC][MT]) {
        // the resource ends after the chunks the count uses: loads of the
        // chunk slots past it return 0 and move no data
        const size_t used = (size_t)((n + 31) / 32) * a.mtiles * 512;
        const __amdgpu_buffer_rsrc_t hr = buf_rsrc(src, (uint32_t)((used < slot_elems ? used : slot_elems) * sizeof(T)));
#pragma unroll
        for (int i = 0; i < MAXC; ++i) {
            const int c = c0 + w + NW * i;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                raw_load<T, CPOL_SC1>(fa[i][mt], hr, m0 + 16 * mt + (lane & 15) < B ? (uint32_t)(frag_lane_off(c, m0 / 16 + mt, lane, a.mtiles) * sizeof(T)) : OOB_OFF);
        }
    };
    // B fragments of the 32-neuron chunk at kc: rows kid[kc..kc+31] of the
    // weight slice Bt (count n; kfull = the contraction length with nothing
    // dropped; bp = the f32 slice's pitch).  Slots past the count read rows
    // of the first chunk (their A side is zero).
    auto load_b = [&](int kc, int n, const int16_t* kid, const T* Bt, int bp, int kfull, Raw8<T> (&fb)[NT]) {
        const int kb = kc < n ? kc : 0;
        if constexpr (KM) {
            // lanes 4e..4e+3 of group g address kept row kb + 8g + e (read 0)
            // and kb + 8g + 4 + e (read 1), at columns 0, 4, 8, 12 of a tile
            const int j = kb + g8 + ((lane & 15) >> 2);
            const T* p0 = Bt + (int)kid[j] * NCP + 4 * (lane & 3);
            const T* p1 = Bt + (int)kid[j + 4] * NCP + 4 * (lane & 3);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const uint2 lo = lds_tr4((const bf16*)(p0 + 16 * nt)), hi = lds_tr4((const bf16*)(p1 + 16 * nt));
                fb[nt].w[0] = lo.x; fb[nt].w[1] = lo.y; fb[nt].w[2] = hi.x; fb[nt].w[3] = hi.y;
            }
        } else if (n == kfull) {                // identity keep list: contiguous rows
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) raw_lds(fb[nt], Bt + (size_t)(nt * 16 + (lane & 15)) * bp + kb + g8);
        } else {
            const int4 k8 = *(const int4*)(kid + kc + g8);          // 8 int16 keep indices
            const int kw[4] = {k8.x, k8.y, k8.z, k8.w};
            int kk[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int j = kc + g8 + e;
                kk[e] = j < n ? (int)(int16_t)(kw[e >> 1] >> (16 * (e & 1))) : 0;
            }
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const T* row = Bt + (size_t)(nt * 16 + (lane & 15)) * bp;
                Frag<T> f;
#pragma unroll
                for (int e = 0; e < 8; ++e) f.v[e] = row[kk[e]];
                raw_from(fb[nt], f);
            }
        }
    };
    // B fragments of round c0
    auto gather_b = [&](int c0, int n, const int16_t* kid, const T* Bt, int bp, int kfull, Raw8<T> (&fbr)[MAXC][NT]) {
#pragma unroll
        for (int i = 0; i < MAXC; ++i) load_b(32 * (c0 + w + NW * i), n, kid, Bt, bp, kfull, fbr[i]);
    };
    // acc += A fragments of round c0 times the B fragments gathered for it
    auto compute_b = [&](Raw8<T> (&fa)[MAXC][MT], const Raw8<T> (&fbr)[MAXC][NT], int c0, int n,
                         f32x4_t (&acc)[MT][NT]) {
#pragma unroll
        for (int i = 0; i < MAXC; ++i) {
            const int kc = 32 * (c0 + w + NW * i);
            if (kc + 32 > n) {                  // last chunk: slots past the keep count hold stale values
                uint32_t m[Raw8<T>::NW];
                pad_mask<T>(kc + g8, n, m);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) raw_and(fa[i][mt], m);
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) raw_mma(fa[i][mt], fbr[i][nt], acc[mt][nt]);
        }
    };
    auto compute = [&](Raw8<T> (&fa)[MAXC][MT], int c0, int n, const int16_t* kid, const T* Bt, int bp, int kfull,
                       f32x4_t (&acc)[MT][NT]) {
#pragma unroll
        for (int i = 0; i < MAXC; ++i) {
            const int kc = 32 * (c0 + w + NW * i);
            Raw8<T> fbr[NT];
            load_b(kc, n, kid, Bt, bp, kfull, fbr);
            if (kc + 32 > n) {                  // last chunk: slots past the keep count hold stale values
                uint32_t m[Raw8<T>::NW];
                pad_mask<T>(kc + g8, n, m);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) raw_and(fa[i][mt], m);
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) raw_mma(fa[i][mt], fbr[nt], acc[mt][nt]);
        }
    };
    auto contract = [&](const T* src, size_t slot_elems, int n, const int16_t* kid, const T* Bt, int bp, int kfull,
                        f32x4_t (&acc)[MT][NT]) {
        for (int c0 = 0; c0 < (n + 31) / 32; c0 += NW * MAXC) {
            Raw8<T> fa[MAXC][MT];
            issue(src, slot_elems, n, c0, fa);
            __builtin_amdgcn_sched_barrier(0);  // every load before the first product
            compute(fa, c0, n, kid, Bt, bp, kfull, acc);
        }
    };

    // Input product of step s (a worker, or a layer that forms its own at
    // the end of the step before, off its recurrence's path): x_t, which the
    // layer below published, times the W-slice rows of the step's keep list,
    // into accx.  The wait skip uses a register copy of the counter taken
    // after the wait's barrier: every thread takes the same branch.  Returns
    // false when a barrier wait failed.
    f32x4_t accx[MT][NT];
    auto x_product = [&](int s) -> bool {
        commit_kidx_x();
        if (seen_dep < (unsigned)(s + 2)) {
            if (!grid_wait(bar_dep, D.dep, nslot, (unsigned)(s + 2), a.err, a.timeout, STATUS_FWD, &dep_seen)) return false;
            seen_dep = dep_seen;
        } else {
            __syncthreads();                    // the keep list just committed
        }
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) accx[i][j] = f32x4_t{0, 0, 0, 0};
        contract((const T*)D.xin + (size_t)step_t(s) * a.xxs, a.xxs, cnt_x, kidx_x, Wt, KP, kin, accx);
        return true;
    };
    // this thread's sums over the waves' partial products (in red) of the
    // four gates of pair q
    auto red_sum = [&](int q, float* pre) {
        const int rr = pb[q] - m0, uu = pu[q] - u0;
        const float* r = red + rr * NC + (uu >> 2) * 16 + (uu & 3) * 4;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const float4 x = *(const float4*)(r + i * MG * NC);
            v.x += x.x; v.y += x.y; v.z += x.z; v.w += x.w;
        }
        pre[0] = v.x; pre[1] = v.y; pre[2] = v.z; pre[3] = v.w;
    };
    auto red_store = [&](f32x4_t (&acc)[MT][NT]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    red[(w * MG + mt * 16 + acc_row(lane, r)) * NC + nt * 16 + (lane & 15)] = acc[mt][nt][r];
        __syncthreads();
    };

    if (worker) {
        // gx_t = s_nr * x~_t W + b for every step, published as soon as x_t is
        prefetch(0);
        for (int s = 0; s < T_; ++s) {
            const int t = step_t(s);
            if (!x_product(s)) break;
            red_store(accx);
#pragma unroll
            for (int q = 0; q < PPT; ++q) {
                const int b = pb[q], u = pu[q];
                if (b >= B || u >= H) continue;
                float pre[4];
                red_sum(q, pre);
#pragma unroll
                for (int g = 0; g < 4; ++g) xstore(D.gxo + ((size_t)t * B + b) * G + g * H + u, D.s_nr * pre[g] + biasr[q][g]);
            }
            prefetch(s + 1);
            grid_arrive(bar);                   // (also: every wave is past its reads of red)
        }
        grid_exit(a.bar, a.nslots, a.err);
        return;
    }

    // prologue: h0 compacted by the keep list of the first step
    const int tfirst = step_t(0);
    {
        const int32_t* pos = D.rh.pos + (size_t)tfirst * D.rh.kmax;
        const uint8_t* msk = D.rh.mask + (size_t)tfirst * D.rh.kmax;
        T* hx0 = (T*)D.hx;
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            if (pb[q] < B && pu[q] < H) {
                const int pp = pos[pu[q]];
                if (pp >= 0)
                    xstore(hx0 + frag_off(pb[q], pp, a.mtiles),
                           (a.dense && !msk[pu[q]]) ? zero_val<T>() : from_f32<T>(hreg[q]));
            }
        }
    }
    prefetch(0);
    grid_arrive(bar);

    const size_t hxs = (size_t)((H + 31) / 32) * a.mtiles * 512;     // elements per h slot
    const bool x_ok = !has_x || x_product(0);
    for (int s = 0; s < T_ && x_ok; ++s) {
        const int t = step_t(s);
        // ---- this step's keep list
        commit_kidx();
        // when the contraction takes one round, its B fragments (U rows
        // through this step's keep list) are read from LDS before the wait
        const bool one_round = cnt <= 32 * NW * MAXC;
        Raw8<T> bh[MAXC][NT];
        if (one_round) {
            __syncthreads();                    // the keep list just committed
            gather_b(0, cnt, kidx, Ut, HP, H, bh);
        }
        // h_{t-1} of every workgroup of this slot, and (a fed layer) the input
        // product of t, whose loads then overlap the product below
        const bool need_dep = fed && seen_dep < (unsigned)(s + 1);
        if (!grid_wait(bar, d, nslot, (unsigned)(s + 1), a.err, a.timeout, STATUS_FWD, nullptr, need_dep ? bar_dep : nullptr,
                       D.dep, (unsigned)(s + 1), &dep_seen))
            break;
        if (need_dep) seen_dep = dep_seen;
        if (fed) load_gx(t);
        f32x4_t acc[MT][NT];
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
        const T* hsrc = (const T*)D.hx + (size_t)(s & 1) * hxs;
        if (one_round) {
            Raw8<T> fh[MAXC][MT];
            issue(hsrc, hxs, cnt, 0, fh);
            __builtin_amdgcn_sched_barrier(0);  // every load before the first product
            compute_b(fh, bh, 0, cnt, acc);
        } else {
            contract(hsrc, hxs, cnt, kidx, Ut, HP, H, acc);
        }
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    acc[i][j][r] = has_x ? D.s_rh * acc[i][j][r] + D.s_nr * accx[i][j][r] : D.s_rh * acc[i][j][r];
        red_store(acc);
        // ---- pointwise (Eq. 1-6); h_t (and the layer above's x_t) is published first
        T* hxn = (T*)D.hx + (size_t)((s + 1) & 1) * hxs;
        float og4[PPT][4], cnv[PPT], hnv[PPT];
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int b = pb[q], u = pu[q];
            if (b >= B || u >= H) continue;
            float pre[4];
            red_sum(q, pre);
#pragma unroll
            for (int g = 0; g < 4; ++g) pre[g] += has_x ? biasr[q][g] : gxr[q][g];
            og4[q][0] = sigmoid_fast(pre[0]);
            og4[q][1] = sigmoid_fast(pre[1]);
            og4[q][2] = tanh_fast(pre[2]);
            og4[q][3] = sigmoid_fast(pre[3]);
            const float cp = creg[q];
            cnv[q] = og4[q][1] * cp + og4[q][0] * og4[q][2];
            hnv[q] = og4[q][3] * tanh_fast(cnv[q]);
            const bool vq = is_valid(q, t);
            const T hv = from_f32<T>(vq ? hnv[q] : hreg[q]);
            // (coherent buffer stores at 32-bit offsets, as xstore)
            if (pn[q] >= 0)
                store_coherent(hxn, hxs, (uint32_t)frag_off(b, pn[q], a.mtiles), (a.dense && !mnr[q]) ? zero_val<T>() : hv);
            if (D.xout && pup[q] >= 0) {
                const T yv = (vq && !(a.dense && !mup[q])) ? from_f32<T>(hnv[q]) : zero_val<T>();
                store_coherent((T*)D.xout + (size_t)t * a.xxs, a.xxs, (uint32_t)frag_off(b, pup[q], a.mtiles), yv);
            }
        }
        grid_arrive(bar);
        // outputs only later kernels read, and the next step's inputs, go out
        // while the other workgroups finish the step
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int b = pb[q], u = pu[q];
            if (b >= B || u >= H) continue;
            const bool vq = is_valid(q, t);
            const float cp = creg[q], cn = vq ? cnv[q] : cp, hn = hnv[q];
            const T hv = from_f32<T>(vq ? hn : hreg[q]);
            *(float4*)(D.gates + ((size_t)t * B + b) * G + 4 * u) = make_float4(og4[q][0], og4[q][1], og4[q][2], og4[q][3]);
            D.cres[((size_t)t * B + b) * H + u] = cn;
            if (vq) { creg[q] = cnv[q]; hreg[q] = hn; }
            ((T*)D.hrecT)[((size_t)t * H + u) * a.BP + b] = hv;
            if (D.y) D.y[((size_t)t * B + b) * a.ldy + u] = vq ? hn : 0.0f;
            if (D.ybuf) {
                const T yv = vq ? from_f32<T>(hn) : zero_val<T>();
                ((T*)D.ybuf)[((size_t)t * B + b) * a.ldy + u] = yv;
                ((T*)D.ybufT)[((size_t)t * a.ldy + u) * a.BP + b] = yv;
            }
        }
        prefetch(s + 1);
        if (has_x && s + 1 < T_ && !x_product(s + 1)) break;
    }
    // ---- final state (NaN if the barrier timed out, and then also every
    // step of the top layer's output)
    const bool failed = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        if (pb[q] < B && pu[q] < H) {
            D.hT[(size_t)pb[q] * H + pu[q]] = failed ? __builtin_nanf("") : hreg[q];
            D.cT[(size_t)pb[q] * H + pu[q]] = failed ? __builtin_nanf("") : creg[q];
            if (failed && D.y)
                for (int t = 0; t < T_; ++t) D.y[((size_t)t * B + pb[q]) * a.ldy + pu[q]] = __builtin_nanf("");
        }
    }
    grid_exit(a.bar, a.nslots, a.err);
}

// ---------------------------------------------------------------------------
// Persistent BPTT (Eq. 7-10).  A launch runs every step of its slots: the
// two directions of one layer, or the layers of a unidirectional stack
// together with one input-gradient worker between each pair of layers (the
// top layer works on step t, the worker below it forms that layer's dx_t from
// the published DA_t, and the next layer uses it one step later).
// Workgroup w -> (slot, unit tile of UB units, row group of MG rows).
// 1024 threads = 16 waves.  Per step: the recurrent gradient of the tile's
// units from DA of the step processed before (Eq. 10; contraction over 4H
// split over the waves; skipped when every unit of the tile was dropped),
// then the pointwise backward (Eq. 7-9) with the dc and pass-through
// carries held in registers.  Dynamic LDS: U rows [UB][GP] (dtype),
// reduction [16][MG][16] (float).  MC: chunks per wave per round, the
// fewest that cover 4H in one round within the register budget (the loads
// of a round are all in flight at once).
constexpr int PB_NW = 16;

template <typename T, int UB, int MG, int MC>
__global__ void __launch_bounds__(1024) k_bwd_persist(PBwdArgs a) {
    constexpr int MT = MG / 16, NW = PB_NW, NTH = 64 * NW;
    constexpr int PPT = (MG * UB + NTH - 1) / NTH;
    constexpr int MAXC = MC;
    extern __shared__ __align__(16) char smem[];
    const int H = a.H, G = 4 * H, B = a.B, T_ = a.T;
    const int GP = (G + 31) / 32 * 32 + 8;       // row pitch; zero past 4H up to the last chunk
    T* Ur = (T*)smem;                                            // [UB][GP]
    float* red = (float*)(smem + (((size_t)UB * GP * sizeof(T) + 15) & ~(size_t)15));

    const int nslot = a.ntiles * a.mgroups;
    const int d = blockIdx.x / nslot, rem = blockIdx.x % nslot;
    const int tile = rem / a.mgroups, mg = rem % a.mgroups;
    const PBwdDir& D = a.d[d];
    const size_t das = (size_t)((G + 31) / 32) * a.mtiles * 512;   // fragment-major DA block per step
    const int u0 = tile * UB, m0 = mg * MG;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int g8 = 8 * (lane >> 4);
    unsigned* bar = slot_bar(a.bar, d);
    const bool worker = D.role == 1;

    // rows of U (a worker: of the input weights of the layer above) for the
    // tile's units -> LDS (zero past 4H and past H)
    // (each thread issues its loads in batches before storing any: a loop
    // of load-then-store waits a full memory latency per element)
    {
        constexpr int LB = 16;
        const T* U = (const T*)(worker ? D.Wup : D.U);
        const int total = UB * GP;
        for (int i0 = tid; i0 < total; i0 += NTH * LB) {
            T v[LB];
#pragma unroll
            for (int j = 0; j < LB; ++j) {
                const int i = min(i0 + NTH * j, total - 1);
                const int r = i / GP, n = i % GP;
                v[j] = U[(size_t)min(u0 + r, H - 1) * G + min(n, G - 1)];
            }
#pragma unroll
            for (int j = 0; j < LB; ++j) {
                const int i = i0 + NTH * j;
                if (i < total) {
                    const int r = i / GP, n = i % GP;
                    Ur[i] = (u0 + r < H && n < G) ? v[j] : zero_val<T>();
                }
            }
        }
    }
    // this thread's (row, unit) pairs and their carries
    float dcs[PPT], dhc[PPT];
    int pb[PPT], pu[PPT];
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        const int p = tid + NTH * q;
        pb[q] = (p < MG * UB) ? m0 + p / UB : B;
        pu[q] = u0 + p % UB;
        const bool ok = pb[q] < B && pu[q] < H;
        dhc[q] = (ok && D.dhT) ? D.dhT[(size_t)pb[q] * H + pu[q]] : 0.f;
        dcs[q] = (ok && D.dcT) ? D.dcT[(size_t)pb[q] * H + pu[q]] : 0.f;
    }
    // per-step inputs (independent of the recurrence), loaded one step ahead
    // from clamped (valid) addresses without branches; the pointwise uses
    // them only for valid (row, unit) pairs.  For iteration s: the inputs of
    // step t(s), and the masks of the tile's units at the step processed
    // before it (whether the tile gets a recurrent gradient, Eq. 10).
    float gt4[PPT][4], ctv[PPT], cpv[PPT], dyr[PPT], dxv[PPT];
    int lenr[PPT], dxp[PPT], mkr[PPT];
    auto step_t = [&](int s) { return D.dir == 0 ? T_ - 1 - s : s; };
    auto prefetch = [&](int s) {
        const int t = step_t(min(s, T_ - 1));
        const int tp = D.dir == 0 ? t - 1 : t + 1;        // forward predecessor of t
        const int tn = step_t(max(s - 1, 0));
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int bc = min(pb[q], B - 1), uc = min(pu[q], H - 1);
            lenr[q] = a.lengths ? a.lengths[bc] : T_;
            const float4 gr = *(const float4*)(D.gates + ((size_t)t * B + bc) * G + 4 * uc);
            gt4[q][0] = gr.x; gt4[q][1] = gr.y; gt4[q][2] = gr.z; gt4[q][3] = gr.w;
            ctv[q] = D.cres[((size_t)t * B + bc) * H + uc];
            cpv[q] = *(s >= T_ - 1 ? D.c0 + (size_t)bc * H + uc : D.cres + ((size_t)tp * B + bc) * H + uc);
            if (D.dy) dyr[q] = D.dy[((size_t)t * B + bc) * a.ldy + uc];
            else if (D.dxc) dxp[q] = D.dxpos[(size_t)t * a.kmax + uc];
            mkr[q] = D.rh.mask[(size_t)tn * a.kmax + uc];
        }
    };
    // the layer above's input gradient: at its compact position (a load that
    // depends on dxp), or from the worker of a stack; issued right after the
    // barrier, beside the DA loads
    auto fetch_dx = [&](int t) {
        if (D.dxw) {
#pragma unroll
            for (int q = 0; q < PPT; ++q) dxv[q] = xload1(D.dxw + ((size_t)t * B + min(pb[q], B - 1)) * H + min(pu[q], H - 1));
            return;
        }
        if (D.dy || !D.dxc) return;
#pragma unroll
        for (int q = 0; q < PPT; ++q)
            dxv[q] = D.dxc[((size_t)t * B + min(pb[q], B - 1)) * a.lddx + max(dxp[q], 0)];
    };
    // whether the tile has a unit kept at the step processed before (the
    // recurrent gradient of a dropped unit is exactly zero); a wave covers
    // every unit of the tile
    auto tile_any_kept = [&]() {
        return __builtin_amdgcn_ballot_w64(pu[0] < H && mkr[0] != 0) != 0;
    };

    // the gradient of the tile's units (Eq. 10) from DA of step tn (of this
    // slot, or of src for a worker) into red
    auto recurrent_product = [&](int tn, const void* da_base) {
        // DA_t is fragment-major: lanes of rows past B read zeros (the cache
        // lines that hold only such rows are not fetched); the columns past
        // 4H of the last chunk are zero (cleared before the backward pass)
        const __amdgpu_buffer_rsrc_t dr = buf_rsrc((const T*)da_base + (size_t)tn * das, (uint32_t)(das * sizeof(T)));
        f32x4_t acc[MT];
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[i] = f32x4_t{0, 0, 0, 0};
        const int nch = (G + 31) / 32;
        const int ul = lane & 15;
        // byte offset of this lane's fragment of tile mt in chunk 0 (out of
        // range for rows past B); chunk c adds c * cbytes
        const uint32_t cbytes = (uint32_t)(a.mtiles * 512 * sizeof(T));
        uint32_t lofs[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            lofs[mt] = m0 + 16 * mt + ul < B ? (uint32_t)(frag_lane_off(0, m0 / 16 + mt, lane, a.mtiles) * sizeof(T)) : OOB_OFF;
        for (int c0 = 0; c0 < nch; c0 += NW * MAXC) {
            Raw8<T> fa[MAXC][MT];
#pragma unroll
            for (int i = 0; i < MAXC; ++i) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) raw_load<T, CPOL_SC1>(fa[i][mt], dr, lofs[mt] + (uint32_t)(c0 + w + NW * i) * cbytes);
            }
            // every load of the round is issued before the first product
            // (the scheduler would otherwise interleave them and pay the
            // memory latency several times)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < MAXC; ++i) {
                const int n = 32 * (c0 + w + NW * i);
                if (n >= G) break;
                Raw8<T> fb;
                raw_lds(fb, Ur + (size_t)ul * GP + n + g8);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) raw_mma(fa[i][mt], fb, acc[mt]);
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int r = 0; r < 4; ++r) red[(w * MG + mt * 16 + acc_row(lane, r)) * 16 + (lane & 15)] = acc[mt][r];
        __syncthreads();
    };
    auto reduced = [&](int rr, int i) {
        float v = 0.f;
#pragma unroll
        for (int q = 0; q < NW; ++q) v += red[(q * MG + rr) * 16 + i];
        return v;
    };

    if (worker) {
        // dx_t of the layer above restricted to this tile's inputs, for every
        // t in that layer's order, as soon as its DA_t is published
        const PBwdDir& S = a.d[D.src];
        unsigned* bar_src = slot_bar(a.bar, D.src);
        for (int s = 0; s < T_; ++s) {
            const int t = step_t(s);
            int mk[PPT];
#pragma unroll
            for (int q = 0; q < PPT; ++q) mk[q] = D.nr_up.mask[(size_t)t * D.nr_up.kmax + min(pu[q], H - 1)];
            if (!grid_wait(bar_src, D.src, nslot, (unsigned)(s + 1), a.err, a.timeout, STATUS_BWD)) break;
            recurrent_product(t, S.da);
#pragma unroll
            for (int q = 0; q < PPT; ++q) {
                const int b = pb[q], u = pu[q];
                if (b >= B || u >= H) continue;
                // dropped inputs get no gradient (output sparsity, Eq. 10)
                const float v = mk[q] ? D.s_nr * reduced(b - m0, u - u0) : 0.0f;
                xstore(D.dxw_out + ((size_t)t * B + b) * H + u, v);
            }
            grid_arrive(bar);
        }
        grid_exit(a.bar, a.nslots, a.err);
        return;
    }

    unsigned* bar_above = D.above >= 0 ? slot_bar(a.bar, D.above) : nullptr;
    __shared__ unsigned above_seen;               // steps of the worker last seen complete
    unsigned seen_above = 0;                      // its copy in every thread (uniform waits)
    prefetch(0);
    for (int s = 0; s <= T_; ++s) {
        const bool final_pass = s == T_;
        const int t = final_pass ? -1 : step_t(s);
        const int tn = D.dir == 0 ? T_ - s : s - 1;        // step processed just before
        const bool has_next = s > 0;
        // DA of the step before from every workgroup of this slot, and the
        // worker's dx of step s (unless a count read earlier covers it), in
        // one wait
        const bool kept = has_next && tile_any_kept();
        const bool need_above = !final_pass && bar_above && seen_above < (unsigned)(s + 1);
        if (has_next || need_above) {
            if (!grid_wait(bar, d, nslot, has_next ? (unsigned)s : 0u, a.err, a.timeout, STATUS_BWD, nullptr,
                           need_above ? bar_above : nullptr, D.above, (unsigned)(s + 1), &above_seen))
                break;
            if (need_above) seen_above = above_seen;
        }
        if (!final_pass) fetch_dx(t);
        if (kept) recurrent_product(tn, D.da);
        float da4[PPT][4];
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
#pragma unroll
            for (int g = 0; g < 4; ++g) da4[q][g] = 0.f;
            const int b = pb[q], u = pu[q];
            if (b >= B || u >= H) continue;
            float dh = dhc[q];
            if (kept) {
                // units dropped at step tn get no recurrent gradient (output sparsity, Eq. 10)
                const float sc = mkr[q] ? D.s_rh : 0.0f;
                dh += sc * reduced(b - m0, u - u0);
            }
            if (final_pass) {
                D.dh0[(size_t)b * H + u] = dh;
                D.dc0[(size_t)b * H + u] = dcs[q];
                continue;
            }
            if (t < lenr[q]) {
                dh += D.dy ? dyr[q] : D.dxw ? dxv[q] : (D.dxc && dxp[q] >= 0 ? dxv[q] : 0.0f);
                const float ig = gt4[q][0], fg = gt4[q][1], gg = gt4[q][2], og = gt4[q][3];
                const float tc = tanh_fast(ctv[q]);
                const float dout = dh * tc;                            // Eq. 7
                const float dc = dh * og * (1.0f - tc * tc) + dcs[q];  // Eq. 7
                da4[q][0] = dc * gg * ig * (1.0f - ig);                // Eq. 9, sigmoid'
                da4[q][1] = dc * cpv[q] * fg * (1.0f - fg);            // Eq. 8, sigmoid'
                da4[q][2] = dc * ig * (1.0f - gg * gg);                // Eq. 9, tanh'
                da4[q][3] = dout * og * (1.0f - og);                   // Eq. 7, sigmoid'
                dcs[q] = dc * fg;                                      // Eq. 8
                dhc[q] = 0.0f;
            } else {
                dhc[q] = dh;                                           // frozen row: pass through
            }
            // coherent stores (SC1, as xstore) through the step's block with
            // 32-bit offsets: a 64-bit element address kept across the step
            // had been spilled to scratch and reloaded here, on the path to
            // the arrival
            const __amdgpu_buffer_rsrc_t dw = buf_rsrc((const T*)D.da + (size_t)t * das, (uint32_t)(das * sizeof(T)));
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const uint32_t o = (uint32_t)frag_off(b, g * H + u, a.mtiles) * (uint32_t)sizeof(T);
                if constexpr (sizeof(T) == 2)
                    __builtin_amdgcn_raw_buffer_store_b16(from_f32<T>(da4[q][g]), dw, o, 0, CPOL_SC1);
                else
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(da4[q][g]), dw, o, 0, CPOL_SC1);
            }
        }
        if (final_pass) break;
        grid_arrive(bar);                                  // DA_t is published
        // the outputs only later kernels read, and the next step's inputs,
        // go out while the other workgroups finish the step.  DA^T (for the
        // weight gradients) is staged in LDS as the tile's [4*UB][MG] block
        // (the reduction area is free until the next step's product; rows
        // past B hold zeros) and written as whole 16-byte pieces of its rows.
        {
            T* st = (T*)red;
#pragma unroll
            for (int q = 0; q < PPT; ++q) {
                const int p = tid + NTH * q;
                if (p >= MG * UB) continue;
                const bool ok = pb[q] < B && pu[q] < H;
#pragma unroll
                for (int g = 0; g < 4; ++g) st[(g * UB + p % UB) * MG + p / UB] = from_f32<T>(ok ? da4[q][g] : 0.f);
            }
            __syncthreads();
            constexpr int PPR = MG * (int)sizeof(T) / 16;  // 16-byte pieces of a staged row
            T* dat = (T*)D.daT + (size_t)t * G * a.BP;
            for (int i = tid; i < 4 * UB * PPR; i += NTH) {
                const int r = i / PPR, pc = i % PPR;
                const int u = u0 + r % UB, col = m0 + pc * (16 / (int)sizeof(T));
                if (u < H && col < a.BP)
                    *(uint4*)(dat + (size_t)((r / UB) * H + u) * a.BP + col) = *(const uint4*)(st + r * MG + pc * (16 / (int)sizeof(T)));
            }
        }
        prefetch(s + 1);
    }
    // a timed-out barrier, here or in the forward pass of the step, poisons
    // the input-state gradients
    if (__hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
        __hip_atomic_load(sync_status(a.err), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
#pragma unroll
        for (int q = 0; q < PPT; ++q)
            if (pb[q] < B && pu[q] < H) {
                D.dh0[(size_t)pb[q] * H + pu[q]] = __builtin_nanf("");
                D.dc0[(size_t)pb[q] * H + pu[q]] = __builtin_nanf("");
            }
    }
    grid_exit(a.bar, a.nslots, a.err);
}

// ---------------------------------------------------------------------------
// Persistent forward recurrence for large batches (Eq. 1-6), one layer (its
// directions as slots).  At a batch where the row-group tiling of
// k_fwd_persist does not fit the device at once (each of its workgroups
// holds a U slice in LDS for every 64 rows), this kernel holds the U slice
// in registers instead and gives LDS to the reduction:
//   workgroup = (slot, 16 hidden units = 64 gate columns, 64 batch rows),
//   512 threads = 8 waves.  Wave w owns the recurrent neurons
//   [32*KC*w, 32*KC*(w+1)) of the contraction: its B fragments (U rows of
//   those neurons, the 64 columns of the tile: KC chunks x 4 column tiles)
//   are loaded once and stay in registers for the whole sequence.  Per step
//   each wave loads the A fragments of its neuron range for the 64 rows
//   (every element of h_{t-1} the workgroup needs is loaded by exactly one
//   wave), forms a 64 x 64 partial product, and the eight partials are
//   summed through LDS by the threads of the gate pointwise (two
//   (row, unit) pairs each).
// h_{t-1} is exchanged uncompacted and multiplied by the step's RH mask at
// the producer (a dropped neuron contributes an exact zero), so the same
// kernel serves both modes; rows and neurons past the shape read as zero.
constexpr int BG_NW = 8, BG_MG = 64, BG_UT = 16, BG_NC = 4 * BG_UT, BG_RP = BG_NC + 4;

template <int KC>
__global__ void __launch_bounds__(512) k_fwd_big(PFwdArgs a) {
    constexpr int MT = BG_MG / 16, NTL = BG_NC / 16, NTH = 64 * BG_NW;
    constexpr int PPT = BG_MG * BG_UT / NTH;   // (row, unit) pairs per thread
    extern __shared__ __align__(16) char smem[];
    float* red = (float*)smem;                 // [8 waves][64 rows][BG_RP]
    const int H = a.H, G = 4 * H, B = a.B, T_ = a.T;
    const int nslot = a.ntiles * a.mgroups;
    const int d = blockIdx.x / nslot, rem = blockIdx.x % nslot;
    const int tile = rem / a.mgroups, mg = rem % a.mgroups;
    const PFwdDir& D = a.d[d];
    const int u0 = tile * BG_UT, m0 = mg * BG_MG;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g8 = 8 * (lane >> 4);
    unsigned* bar = slot_bar(a.bar, d);
    const int nch = (H + 31) / 32;             // 32-neuron chunks of the contraction

    // B fragments: U rows of this wave's neurons, the tile's 64 columns
    // (column c of tile j is gate (c&15)>>2 of unit u0 + 4j + (c&3))
    bf16x8_t ub[KC][NTL];
    {
        const bf16* U = (const bf16*)D.U;
#pragma unroll
        for (int j = 0; j < NTL; ++j) {
            const int cl = lane & 15;
            const int unit = u0 + 4 * j + (cl & 3);
            const int gcol = (cl >> 2) * H + min(unit, H - 1);
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                const int kb = 32 * (w * KC + c) + g8;
                s16x8_t f;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int k = kb + e;
                    const bf16 v = U[(size_t)min(k, H - 1) * G + gcol];
                    f[e] = (short)((k < H && unit < H) ? v : (bf16)0);
                }
                ub[c][j] = __builtin_bit_cast(bf16x8_t, f);
            }
        }
    }
    // this thread's (row, unit) pairs, their state and per-step inputs
    float creg[PPT], hreg[PPT], gxr[PPT][4];
    int pb[PPT], pu[PPT], lenr[PPT], mnx[PPT];
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        const int p = tid + NTH * q;
        pb[q] = m0 + p / BG_UT;
        pu[q] = u0 + p % BG_UT;
        const bool ok = pb[q] < B && pu[q] < H;
        creg[q] = ok ? D.c0[(size_t)pb[q] * H + pu[q]] : 0.f;
        hreg[q] = ok ? bf2f(((const bf16*)D.h0)[(size_t)pb[q] * H + pu[q]]) : 0.f;
        lenr[q] = a.lengths ? a.lengths[min(pb[q], B - 1)] : T_;
    }
    auto step_t = [&](int s) { return D.dir == 0 ? s : T_ - 1 - s; };
    // inputs of step s (clamped, valid addresses): the input product and the
    // RH mask of the step that consumes h_t
    auto prefetch = [&](int s) {
        const int sc = min(s, T_ - 1);
        const int t = step_t(sc);
        const int tn = step_t(min(sc + 1, T_ - 1));
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int bc = min(pb[q], B - 1), uc = min(pu[q], H - 1);
            const float* gp = D.gx + ((size_t)t * B + bc) * G + uc;
#pragma unroll
            for (int g = 0; g < 4; ++g) gxr[q][g] = gp[g * H];
            mnx[q] = D.rh.mask[(size_t)tn * D.rh.kmax + uc];
        }
    };
    const size_t hxs = (size_t)nch * a.mtiles * 512;       // elements per h slot
    // this lane's A offset in chunk 0 of the wave and row tile 0 of the group
    const uint32_t a_base = (uint32_t)(frag_lane_off(w * KC, m0 / 16, lane, a.mtiles) * sizeof(bf16));
    // Rows past the batch inside its last 16-row tile are never written and
    // only reach outputs of rows past the batch (not stored).  Neurons past H
    // in the last chunk are never written either and meet zero U rows, so
    // they are cleared here, in both slots, before the first barrier (a
    // stale NaN times zero would not vanish): the last unit tile's
    // workgroups clear them for their rows.
    if (tile == a.ntiles - 1 && H % 32) {
        const int npad = 32 * nch - H;
        for (int i = tid; i < 2 * BG_MG * npad; i += NTH) {
            const int sl = i / (BG_MG * npad), r = (i / npad) % BG_MG, k = H + i % npad;
            if (m0 + r < 16 * a.mtiles)
                xstore((bf16*)D.hx + (size_t)sl * hxs + frag_off(m0 + r, k, a.mtiles), (bf16)0);
        }
    }
    // prologue: h0 times the first step's RH mask into slot 0
    {
        const int t0 = step_t(0);
        bf16* hx0 = (bf16*)D.hx;
#pragma unroll
        for (int q = 0; q < PPT; ++q)
            if (pb[q] < B && pu[q] < H)
                xstore(hx0 + frag_off(pb[q], pu[q], a.mtiles),
                       D.rh.mask[(size_t)t0 * D.rh.kmax + pu[q]] ? f2bf(hreg[q]) : (bf16)0);
    }
    prefetch(0);
    grid_arrive(bar);

    for (int s = 0; s < T_; ++s) {
        const int t = step_t(s);
        if (!grid_wait(bar, d, nslot, (unsigned)(s + 1), a.err, a.timeout, STATUS_FWD)) break;
        // ---- h~_{t-1} (this wave's neurons, the tile's rows) times the U slice
        // A fragments two chunks deep (registers): chunk c+2 is issued as
        // soon as chunk c has been multiplied.  Offsets: one base register
        // (copied inside the loop, so the compiler keeps one register rather
        // than hoisting a register per fragment) plus the chunk; the row tile
        // is the instruction's immediate (tiles are 1 KB apart).  Chunks past
        // the last one and row tiles past the last one of the batch read
        // past the slot (zero) or rows past the batch (whose outputs are not
        // stored).
        const __amdgpu_buffer_rsrc_t hr = buf_rsrc((const bf16*)D.hx + (size_t)(s & 1) * hxs,
                                                   (uint32_t)(hxs * sizeof(bf16)));
        uint32_t vb;
        asm volatile("v_mov_b32 %0, %1" : "=v"(vb) : "v"(a_base));
        auto issue = [&](int c, u32x4_t (&f)[MT]) {
            const uint32_t vo = vb + (uint32_t)(c * a.mtiles * 1024);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) f[mt] = __builtin_amdgcn_raw_buffer_load_b128(hr, vo + mt * 1024, 0, CPOL_SC1);
        };
        u32x4_t fa[2][MT];
        issue(0, fa[0]);
        if (KC > 1) issue(1, fa[1]);
        f32x4_t acc[MT][NTL];
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NTL; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            u32x4_t (&f)[MT] = fa[c & 1];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bf16x8_t av = __builtin_bit_cast(bf16x8_t, f[mt]);
#pragma unroll
                for (int j = 0; j < NTL; ++j)
                    acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, ub[c][j], acc[mt][j], 0, 0, 0);
            }
            if (c + 2 < KC) issue(c + 2, f);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int j = 0; j < NTL; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    red[(w * BG_MG + mt * 16 + acc_row(lane, r)) * BG_RP + j * 16 + (lane & 15)] = acc[mt][j][r];
        __syncthreads();
        // ---- pointwise (Eq. 1-6); h_t goes out first, masked for the next step
        bf16* hxn = (bf16*)D.hx + (size_t)((s + 1) & 1) * hxs;
        float og4[PPT][4], cnv[PPT], hnv[PPT];
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int p = tid + NTH * q;
            const int rr = p / BG_UT, uu = p % BG_UT;
            const int cb = (uu >> 2) * 16 + (uu & 3);
            float pre[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                float v = 0.f;
#pragma unroll
                for (int i = 0; i < BG_NW; ++i) v += red[(i * BG_MG + rr) * BG_RP + cb + 4 * g];
                pre[g] = D.s_rh * v + gxr[q][g];
            }
            og4[q][0] = sigmoid_fast(pre[0]);
            og4[q][1] = sigmoid_fast(pre[1]);
            og4[q][2] = tanh_fast(pre[2]);
            og4[q][3] = sigmoid_fast(pre[3]);
            cnv[q] = og4[q][1] * creg[q] + og4[q][0] * og4[q][2];
            hnv[q] = og4[q][3] * tanh_fast(cnv[q]);
            if (pb[q] < B && pu[q] < H && s + 1 < T_) {
                const bool vq = t < lenr[q];
                xstore(hxn + frag_off(pb[q], pu[q], a.mtiles), mnx[q] ? f2bf(vq ? hnv[q] : hreg[q]) : (bf16)0);
            }
        }
        grid_arrive(bar);
        // outputs only later kernels read, and the next step's inputs
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int b = pb[q], u = pu[q];
            if (b >= B || u >= H) continue;
            const bool vq = t < lenr[q];
            const float cn = vq ? cnv[q] : creg[q], hn = hnv[q];
            const bf16 hv = f2bf(vq ? hn : hreg[q]);
            *(float4*)(D.gates + ((size_t)t * B + b) * G + 4 * u) = make_float4(og4[q][0], og4[q][1], og4[q][2], og4[q][3]);
            D.cres[((size_t)t * B + b) * H + u] = cn;
            if (vq) { creg[q] = cnv[q]; hreg[q] = hn; }
            ((bf16*)D.hrecT)[((size_t)t * H + u) * a.BP + b] = hv;
            if (D.y) D.y[((size_t)t * B + b) * a.ldy + u] = vq ? hn : 0.0f;
            if (D.ybuf) {
                const bf16 yv = vq ? f2bf(hn) : (bf16)0;
                ((bf16*)D.ybuf)[((size_t)t * B + b) * a.ldy + u] = yv;
                ((bf16*)D.ybufT)[((size_t)t * a.ldy + u) * a.BP + b] = yv;
            }
        }
        prefetch(s + 1);
    }
    // ---- final state (NaN if a barrier wait timed out, and then every step of y)
    const bool failed = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        if (pb[q] < B && pu[q] < H) {
            D.hT[(size_t)pb[q] * H + pu[q]] = failed ? __builtin_nanf("") : hreg[q];
            D.cT[(size_t)pb[q] * H + pu[q]] = failed ? __builtin_nanf("") : creg[q];
            if (failed && D.y)
                for (int t = 0; t < T_; ++t) D.y[((size_t)t * B + pb[q]) * a.ldy + pu[q]] = __builtin_nanf("");
        }
    }
    grid_exit(a.bar, a.nslots, a.err);
}

// ---------------------------------------------------------------------------
// Persistent BPTT for large batches (Eq. 7-10), one layer.  The recurrent
// gradient of a step, dh_{t-1} = (DA_t U^T) * m * s, is a product over the
// 4H gate columns; at a large batch it runs split over the gate columns so
// that every workgroup keeps a 128-unit x 512-column block of U in
// registers:
//   phase A (pointwise, Eq. 7-9): workgroup = (16 units, 64 rows); sums the
//     partial gradients of the step before over the column groups, forms
//     DA_t of its tile and publishes it;
//   phase B (product, Eq. 10): workgroup = (64 rows, unit group of 128,
//     column group of 512); each wave multiplies 4 of the group's 16
//     column chunks for 64 of its units, the four column quarters are
//     summed through LDS and the group's partial [B][H] is published.
// Two grid barriers per step; partial sums are added in a fixed order.
constexpr int BB_NW = 8, BB_MG = 64, BB_UT = 16, BB_UG = 128, BB_KG = 512, BB_RP = BB_UG + 4;

__global__ void __launch_bounds__(512) k_bwd_big(PBwdArgs a) {
    constexpr int MT = BB_MG / 16, NTH = 64 * BB_NW, KC = 4, NTL = 4;
    constexpr int PPT = BB_MG * BB_UT / NTH;   // (row, unit) pairs per thread in phase A
    extern __shared__ __align__(16) char smem[];
    float* red = (float*)smem;                 // phase B: [4 column quarters][64 rows][BB_RP]
    const int H = a.H, G = 4 * H, B = a.B, T_ = a.T;
    const int nslot = gridDim.x;               // one slot (one direction per launch)
    const PBwdDir& D = a.d[0];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g8 = 8 * (lane >> 4);
    unsigned* bar = slot_bar(a.bar, 0);
    const size_t das = (size_t)((G + 31) / 32) * a.mtiles * 512;   // fragment-major DA block per step
    const int nchG = (G + 31) / 32;

    // ---- phase A role: (unit tile, row group)
    const int nA = a.ntiles * a.mgroups;
    const bool roleA = (int)blockIdx.x < nA;
    const int tA = blockIdx.x / a.mgroups, mA = blockIdx.x % a.mgroups;
    const int u0 = tA * BB_UT, mA0 = mA * BB_MG;
    // ---- phase B role: (row group, unit group, column group)
    const int nB = a.mgroups * a.ngu * a.ngk;
    const bool roleB = (int)blockIdx.x < nB;
    const int rgB = blockIdx.x % a.mgroups, ugB = (blockIdx.x / a.mgroups) % a.ngu,
              kgB = blockIdx.x / (a.mgroups * a.ngu);
    const int mB0 = rgB * BB_MG;
    const int kq = w >> 1, ch = w & 1;         // this wave's column quarter and unit half

    // U block in registers: B fragment (chunk c, unit tile j) of this wave:
    // contraction = gate columns, output columns = units
    bf16x8_t ub[KC][NTL];
    {
        const bf16* U = (const bf16*)D.U;
#pragma unroll
        for (int j = 0; j < NTL; ++j) {
            const int u = BB_UG * ugB + 16 * (NTL * ch + j) + (lane & 15);
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                const int n0 = BB_KG * kgB + 32 * (KC * kq + c) + g8;
                s16x8_t f;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int n = n0 + e;
                    const bf16 v = U[(size_t)min(u, H - 1) * G + min(n, G - 1)];
                    f[e] = (short)((roleB && u < H && n < G) ? v : (bf16)0);
                }
                ub[c][j] = __builtin_bit_cast(bf16x8_t, f);
            }
        }
    }
    // phase A pairs and their carries: pair p = tid + 512q is row p/16 of
    // the group, unit p%16 of the tile (16 lanes on 16 adjacent units)
    float dcs[PPT], dhc[PPT];
    int pb[PPT], pu[PPT], lenr[PPT];
#pragma unroll
    for (int q = 0; q < PPT; ++q) {
        const int p = tid + NTH * q;
        pb[q] = roleA ? mA0 + p / BB_UT : B;
        pu[q] = u0 + p % BB_UT;
        const bool ok = pb[q] < B && pu[q] < H;
        dhc[q] = (ok && D.dhT) ? D.dhT[(size_t)pb[q] * H + pu[q]] : 0.f;
        dcs[q] = (ok && D.dcT) ? D.dcT[(size_t)pb[q] * H + pu[q]] : 0.f;
        lenr[q] = a.lengths ? a.lengths[min(pb[q], B - 1)] : T_;
    }
    auto step_t = [&](int s) { return D.dir == 0 ? T_ - 1 - s : s; };
    // per-step inputs of phase A (clamped addresses), one step ahead
    float gt4[PPT][4], ctv[PPT], cpv[PPT], dyv[PPT];
    int mkr[PPT];
    auto prefetch = [&](int s) {
        const int t = step_t(min(s, T_ - 1));
        const int tp = D.dir == 0 ? t - 1 : t + 1;        // forward predecessor of t
        const int tn = step_t(max(s - 1, 0));              // the step processed before
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
            const int bc = min(pb[q], B - 1), uc = min(pu[q], H - 1);
            const float4 gr = *(const float4*)(D.gates + ((size_t)t * B + bc) * G + 4 * uc);
            gt4[q][0] = gr.x; gt4[q][1] = gr.y; gt4[q][2] = gr.z; gt4[q][3] = gr.w;
            ctv[q] = D.cres[((size_t)t * B + bc) * H + uc];
            cpv[q] = *(s >= T_ - 1 ? D.c0 + (size_t)bc * H + uc : D.cres + ((size_t)tp * B + bc) * H + uc);
            if (D.dy) {
                dyv[q] = D.dy[((size_t)t * B + bc) * a.ldy + uc];
            } else if (D.dxc) {
                const int dp = D.dxpos[(size_t)t * a.kmax + uc];
                dyv[q] = dp >= 0 ? D.dxc[((size_t)t * B + bc) * a.lddx + dp] : 0.0f;
            } else {
                dyv[q] = 0.0f;
            }
            mkr[q] = D.rh.mask[(size_t)tn * a.kmax + uc];
        }
    };
    // this lane's A offset in the wave's first chunk and the group's first
    // row tile (chunks past 4H read past the block: zero)
    const uint32_t a_base = (uint32_t)(frag_lane_off((BB_KG / 32) * kgB + KC * kq, mB0 / 16, lane, a.mtiles) *
                                       sizeof(bf16));

    prefetch(0);
    bool ok = true;
    // hidden sizes in multiples of 8: DA goes out as whole 16-byte pieces
    const bool wide = (H & 7) == 0;
    for (int s = 0; s <= T_; ++s) {
        const bool final_pass = s == T_;
        const int t = final_pass ? -1 : step_t(s);
        // ---- phase A: the partial recurrent gradients of the step before
        // (phase B of iteration s-1) are complete after 2s arrivals
        if (s > 0 && !(ok = grid_wait(bar, 0, nslot, (unsigned)(2 * s), a.err, a.timeout, STATUS_BWD))) break;
        // the recurrent gradients of the thread's pairs: the partial sums of
        // the column groups, 8 groups' loads of both pairs in flight at once
        // (absent groups read group 0; clamped addresses: the results of
        // pairs outside the batch or the layer are not used), added in group
        // order
        float rg[PPT] = {0.f, 0.f};
        if (s > 0) {
            for (int k0 = 0; k0 < a.ngk; k0 += 8) {
                float pv[PPT][8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const float* pk = a.part + (size_t)(k0 + k < a.ngk ? k0 + k : 0) * B * H;
#pragma unroll
                    for (int q = 0; q < PPT; ++q)
                        pv[q][k] = xload1(pk + (size_t)min(pb[q], B - 1) * H + min(pu[q], H - 1));
                }
#pragma unroll
                for (int k = 0; k < 8; ++k)
#pragma unroll
                    for (int q = 0; q < PPT; ++q)
                        if (k0 + k < a.ngk) rg[q] += pv[q][k];
            }
        }
        float da4[PPT][4];
#pragma unroll
        for (int q = 0; q < PPT; ++q) {
#pragma unroll
            for (int g = 0; g < 4; ++g) da4[q][g] = 0.f;
            // (copies the compiler cannot hoist: the addresses derived from
            // them are recomputed per step instead of occupying registers)
            int b = pb[q], u = pu[q];
            asm volatile("" : "+v"(b), "+v"(u));
            if (b >= B || u >= H) continue;
            float dh = dhc[q];
            // units dropped at the step before get no recurrent gradient (Eq. 10)
            if (s > 0 && mkr[q]) dh += D.s_rh * rg[q];
            if (final_pass) {
                D.dh0[(size_t)b * H + u] = dh;
                D.dc0[(size_t)b * H + u] = dcs[q];
                continue;
            }
            if (t < lenr[q]) {
                dh += dyv[q];
                const float ig = gt4[q][0], fg = gt4[q][1], gg = gt4[q][2], og = gt4[q][3];
                const float tc = tanh_fast(ctv[q]);
                const float dout = dh * tc;                            // Eq. 7
                const float dc = dh * og * (1.0f - tc * tc) + dcs[q];  // Eq. 7
                da4[q][0] = dc * gg * ig * (1.0f - ig);                // Eq. 9, sigmoid'
                da4[q][1] = dc * cpv[q] * fg * (1.0f - fg);            // Eq. 8, sigmoid'
                da4[q][2] = dc * ig * (1.0f - gg * gg);                // Eq. 9, tanh'
                da4[q][3] = dout * og * (1.0f - og);                   // Eq. 7, sigmoid'
                dcs[q] = dc * fg;                                      // Eq. 8
                dhc[q] = 0.0f;
            } else {
                dhc[q] = dh;                                           // frozen row: pass through
            }
            if (!wide) {
                bf16* dar = (bf16*)D.da + (size_t)t * das;
#pragma unroll
                for (int g = 0; g < 4; ++g) xstore(dar + frag_off(b, g * H + u, a.mtiles), f2bf(da4[q][g]));
            }
        }
        if (final_pass) break;
        if (wide && roleA) {
            // DA_t of the tile through LDS ([64 rows][4 gates x 16 units]),
            // published as 16-byte pieces: 8 adjacent units of one gate and
            // row are one piece of the fragment-major block
            bf16* st = (bf16*)red;
#pragma unroll
            for (int q = 0; q < PPT; ++q) {
                const int p = tid + NTH * q;
#pragma unroll
                for (int g = 0; g < 4; ++g) st[(p / BB_UT) * 64 + g * BB_UT + p % BB_UT] = f2bf(da4[q][g]);
            }
            __syncthreads();
            const int rr = tid >> 3, g = (tid >> 1) & 3, h = tid & 1;
            const int b = mA0 + rr, uh = u0 + 8 * h;
            if (b < B && uh < H) {
                const __amdgpu_buffer_rsrc_t dw = buf_rsrc((const bf16*)D.da + (size_t)t * das, (uint32_t)(das * 2));
                const u32x4_t v = *(const u32x4_t*)(st + rr * 64 + g * BB_UT + 8 * h);
                __builtin_amdgcn_raw_buffer_store_b128(v, dw, (uint32_t)(frag_off(b, g * H + uh, a.mtiles) * 2), 0, CPOL_SC1);
            }
        }
        grid_arrive(bar);                                  // DA_t is published (arrival 2s+1)
        // DA^T (the weight gradients' operand) through LDS: the tile's
        // [4 gates x 16 units][64 rows] block, written as 16-byte row pieces
        if (roleA) {
            bf16* st = (bf16*)red;
#pragma unroll
            for (int q = 0; q < PPT; ++q) {
                const int p = tid + NTH * q;
                const bool okp = pb[q] < B && pu[q] < H;
#pragma unroll
                for (int g = 0; g < 4; ++g) st[(g * BB_UT + p % BB_UT) * BB_MG + p / BB_UT] = f2bf(okp ? da4[q][g] : 0.f);
            }
            __syncthreads();
            constexpr int PPR = BB_MG * 2 / 16;            // 16-byte pieces of a staged row
            bf16* dat = (bf16*)D.daT + (size_t)t * G * a.BP;
            for (int i = tid; i < 4 * BB_UT * PPR; i += NTH) {
                const int r = i / PPR, pc = i % PPR;
                const int u = u0 + r % BB_UT, col = mA0 + pc * 8;
                if (u < H && col < a.BP)
                    *(uint4*)(dat + (size_t)((r / BB_UT) * H + u) * a.BP + col) = *(const uint4*)(st + r * BB_MG + pc * 8);
            }
        }
        // ---- phase B: every DA_t tile is published after 2s+1 arrivals
        if (!(ok = grid_wait(bar, 0, nslot, (unsigned)(2 * s + 1), a.err, a.timeout, STATUS_BWD))) break;
        if (roleB) {
            // A fragments (DA_t rows of the group, this wave's column quarter)
            // two chunks deep; offsets as in the large-batch forward
            const __amdgpu_buffer_rsrc_t dr = buf_rsrc((const bf16*)D.da + (size_t)t * das,
                                                       (uint32_t)(das * sizeof(bf16)));
            uint32_t vb;
            asm volatile("v_mov_b32 %0, %1" : "=v"(vb) : "v"(a_base));
            auto issue = [&](int c, u32x4_t (&f)[MT]) {
                const uint32_t vo = vb + (uint32_t)(c * a.mtiles * 1024);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    f[mt] = __builtin_amdgcn_raw_buffer_load_b128(dr, vo + mt * 1024, 0, CPOL_SC1);
            };
            u32x4_t fa[2][MT];
            issue(0, fa[0]);
            issue(1, fa[1]);
            f32x4_t acc[MT][NTL];
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < NTL; ++j) acc[i][j] = f32x4_t{0, 0, 0, 0};
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                u32x4_t (&f)[MT] = fa[c & 1];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const bf16x8_t av = __builtin_bit_cast(bf16x8_t, f[mt]);
#pragma unroll
                    for (int j = 0; j < NTL; ++j)
                        acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, ub[c][j], acc[mt][j], 0, 0, 0);
                }
                if (c + 2 < KC) issue(c + 2, f);
            }
            // (the DA^T staging of phase A is done with the LDS area: every
            // thread passed the barrier wait above after its stores)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int j = 0; j < NTL; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        red[(kq * BB_MG + mt * 16 + acc_row(lane, r)) * BB_RP + 64 * ch + 16 * j + (lane & 15)] =
                            acc[mt][j][r];
            __syncthreads();
            float* pk = a.part + (size_t)kgB * B * H;
            if ((H & 3) == 0) {                // four adjacent units, one 16-byte coherent store
                const __amdgpu_buffer_rsrc_t pr = buf_rsrc(pk, (uint32_t)((size_t)B * H * 4));
                for (int i = tid; i < BB_MG * BB_UG / 4; i += NTH) {
                    const int rr = i / (BB_UG / 4), uu = 4 * (i % (BB_UG / 4));
                    const int b = mB0 + rr, u = BB_UG * ugB + uu;
                    if (b < B && u < H) {
                        float4 v = *(const float4*)(red + (size_t)rr * BB_RP + uu);
#pragma unroll
                        for (int k = 1; k < 4; ++k) {
                            const float4 x = *(const float4*)(red + (size_t)(k * BB_MG + rr) * BB_RP + uu);
                            v.x += x.x; v.y += x.y; v.z += x.z; v.w += x.w;
                        }
                        const u32x4_t o = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                                           __float_as_uint(v.w)};
                        __builtin_amdgcn_raw_buffer_store_b128(o, pr, (uint32_t)(((size_t)b * H + u) * 4), 0, CPOL_SC1);
                    }
                }
            } else {
                for (int i = tid; i < BB_MG * BB_UG; i += NTH) {
                    const int rr = i / BB_UG, uu = i % BB_UG;
                    const int b = mB0 + rr, u = BB_UG * ugB + uu;
                    if (b < B && u < H) {
                        float v = 0.f;
#pragma unroll
                        for (int k = 0; k < 4; ++k) v += red[(k * BB_MG + rr) * BB_RP + uu];
                        xstore(pk + (size_t)b * H + u, v);
                    }
                }
            }
        }
        grid_arrive(bar);                                  // the partials are published (arrival 2s+2)
        prefetch(s + 1);                                   // (in flight during the next wait)
    }
    // a timed-out barrier, here or in the forward pass of the step, poisons
    // the input-state gradients
    if (!ok || __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
        __hip_atomic_load(sync_status(a.err), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
#pragma unroll
        for (int q = 0; q < PPT; ++q)
            if (pb[q] < B && pu[q] < H) {
                D.dh0[(size_t)pb[q] * H + pu[q]] = __builtin_nanf("");
                D.dc0[(size_t)pb[q] * H + pu[q]] = __builtin_nanf("");
            }
    }
    grid_exit(a.bar, 1, a.err);
}

// ---------------------------------------------------------------------------
// Host side.

// Checks (once per device, kernel and LDS size) that nwg workgroups of the
// kernel can be resident at once; sets the dynamic LDS limit on first use.
static hipError_t resident_limit(const void* fn, int threads, size_t lds, int nwg) {
    struct Entry { int dev; const void* fn; size_t lds; int max_wg; };
    static std::vector<Entry> cache;
    static std::mutex mu;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    int max_wg = -1;
    for (const Entry& c : cache)
        if (c.dev == dev && c.fn == fn && c.lds == lds) max_wg = c.max_wg;
    if (max_wg < 0) {
        hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        int per_cu = 0, ncu = 0;
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds);
        if (e != hipSuccess) return e;
        if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return hipErrorInvalidDevice;
        max_wg = per_cu * ncu;
        cache.push_back({dev, fn, lds, max_wg});
    }
    return (nwg <= max_wg) ? hipSuccess : hipErrorCooperativeLaunchTooLarge;
}

// The persistent grids fit the device (resident_limit) and the stream runs
// them after the previous kernel has drained, so every workgroup is placed
// at once; a barrier wait is bounded in any case (time-out -> error flag and
// the sticky status word that lstm_sd_status reads).
// LDS layout: U slice at 0; the W slice at wofs (in place of U when only
// workers hold W slices, after U when layers form their own input
// products); keep lists at kofs; then the reduction area.  Returns the size.
size_t fwd_persist_lds(int H, int NT, int MG, int esize, int KP, int kin_max, bool w_beside_u, size_t* wofs,
                       size_t* kofs) {
    const size_t cols = esize == 2 ? (size_t)fwd_ncp(NT) : (size_t)16 * NT;   // bf16: K-major, padded rows
    const size_t us = (cols * fwd_hp(H) * esize + 15) & ~(size_t)15;
    const size_t ws = (cols * KP * esize + 15) & ~(size_t)15;
    *wofs = w_beside_u ? us : 0;
    *kofs = w_beside_u ? us + ws : (us > ws ? us : ws);
    const size_t kx = (size_t)(((H + 32) + 7) & ~7) * 2;
    const size_t kxx = KP ? (((size_t)(kin_max + 32) * 2 + 15) & ~(size_t)15) : 0;
    return *kofs + kx + kxx + (size_t)PF_NW * MG * 16 * NT * 4;
}

// Launches the persistent forward if its grid fits the device at once;
// returns hipSuccess, or an error before anything was enqueued (the caller
// then takes another layout or the per-step kernels).
template <typename T>
hipError_t launch_fwd_persist(PFwdArgs& a, hipStream_t st, int kid_timer_on, hipEvent_t e0, hipEvent_t e1) {
    const int MG = a.B <= 32 ? 32 : 64;
    const int NT = a.H >= 512 ? 2 : 1;  // fewer, wider unit tiles: a cheaper barrier
    a.ntiles = (a.H + 4 * NT - 1) / (4 * NT);
    a.mgroups = (a.B + MG - 1) / MG;
    const int nwg = a.nslots * a.ntiles * a.mgroups;
    bool w_beside_u = false;            // a layer slot forming its own input product holds U and W
    for (int i = 0; i < a.nslots; ++i) w_beside_u = w_beside_u || (a.d[i].role == 0 && a.d[i].Win);
    const size_t lds = fwd_persist_lds(a.H, NT, MG, (int)sizeof(T), a.KP, a.kin_max, w_beside_u, &a.wofs, &a.kofs);
    if (lds > 160 * 1024 || a.nslots > 8) return hipErrorInvalidValue;
    void (*fn)(PFwdArgs) = NT == 1 ? (MG == 32 ? k_fwd_persist<T, 1, 32> : k_fwd_persist<T, 1, 64>)
                                   : (MG == 32 ? k_fwd_persist<T, 2, 32> : k_fwd_persist<T, 2, 64>);
    hipError_t e = resident_limit((const void*)fn, 64 * PF_NW, lds, nwg);
    if (e != hipSuccess) return e;
    if (kid_timer_on) (void)hipEventRecord(e0, st);
    hipLaunchKernelGGL(fn, dim3(nwg), dim3(64 * PF_NW), lds, st, a);
    e = hipGetLastError();
    if (kid_timer_on && e == hipSuccess) (void)hipEventRecord(e1, st);
    return e;
}

template hipError_t launch_fwd_persist<float>(PFwdArgs&, hipStream_t, int, hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_persist<bf16>(PFwdArgs&, hipStream_t, int, hipEvent_t, hipEvent_t);

// The large-batch forward (bf16): returns an error before anything is
// enqueued when the shape is outside its register budget or the grid does
// not fit the device at once.
hipError_t launch_fwd_big(PFwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1) {
    const int KC = a.H <= 512 ? 2 : a.H <= 1024 ? 4 : 0;
    if (!KC || a.nslots > 2) return hipErrorInvalidValue;
    a.ntiles = (a.H + BG_UT - 1) / BG_UT;
    a.mgroups = (a.B + BG_MG - 1) / BG_MG;
    const int nwg = a.nslots * a.ntiles * a.mgroups;
    const size_t lds = (size_t)BG_NW * BG_MG * BG_RP * sizeof(float);
    void (*fn)(PFwdArgs) = KC == 2 ? k_fwd_big<2> : k_fwd_big<4>;
    hipError_t e = resident_limit((const void*)fn, 64 * BG_NW, lds, nwg);
    if (e != hipSuccess) return e;
    if (timer_on) (void)hipEventRecord(e0, st);
    hipLaunchKernelGGL(fn, dim3(nwg), dim3(64 * BG_NW), lds, st, a);
    e = hipGetLastError();
    if (timer_on && e == hipSuccess) (void)hipEventRecord(e1, st);
    return e;
}

size_t bwd_persist_lds(int H, int UB, int MG, int esize) {
    const size_t G = 4 * (size_t)H, GP = (G + 31) / 32 * 32 + 8;
    return (((size_t)UB * GP * esize + 15) & ~(size_t)15) + (size_t)PB_NW * MG * 16 * 4;
}

template <typename T, int UB, int MG, int MC>
static hipError_t launch_bwd_persist_t(const PBwdArgs& a, int nwg, size_t lds, hipStream_t st) {
    auto fn = k_bwd_persist<T, UB, MG, MC>;
    const hipError_t e = resident_limit((const void*)fn, 64 * PB_NW, lds, nwg);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(nwg), dim3(64 * PB_NW), lds, st, a);
    return hipGetLastError();
}

// Launches the persistent backward layer if it fits (else returns an error
// and nothing was launched).
template <typename T>
hipError_t launch_bwd_persist(PBwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1) {
    const int MG = a.B <= 32 ? 32 : 64;
    a.mgroups = (a.B + MG - 1) / MG;
    int UB = 16;
    if (bwd_persist_lds(a.H, 16, MG, (int)sizeof(T)) > 160 * 1024) UB = 8;
    const size_t lds = bwd_persist_lds(a.H, UB, MG, (int)sizeof(T));
    if (lds > 160 * 1024) return hipErrorInvalidValue;
    a.ntiles = (a.H + UB - 1) / UB;
    const int nwg = a.nslots * a.ntiles * a.mgroups;
    if (a.nslots > 8) return hipErrorInvalidValue;
    if (timer_on) (void)hipEventRecord(e0, st);
    // chunks per wave per round: 128 VGPRs at 1024 threads hold 6 bf16
    // rounds of 32-row fragments (3 f32), 2 of 64-row ones (1 f32)
    const int nch = (4 * a.H + 31) / 32, per_wave = (nch + PB_NW - 1) / PB_NW;
    hipError_t e;
    if constexpr (sizeof(T) == 4) {
        if (UB == 16) e = MG == 32 ? launch_bwd_persist_t<T, 16, 32, 3>(a, nwg, lds, st)
                                   : launch_bwd_persist_t<T, 16, 64, 1>(a, nwg, lds, st);
        else e = MG == 32 ? launch_bwd_persist_t<T, 8, 32, 3>(a, nwg, lds, st)
                          : launch_bwd_persist_t<T, 8, 64, 1>(a, nwg, lds, st);
    } else if (MG == 64) {
        e = UB == 16 ? launch_bwd_persist_t<T, 16, 64, 2>(a, nwg, lds, st)
                     : launch_bwd_persist_t<T, 8, 64, 2>(a, nwg, lds, st);
    } else if (per_wave <= 2) {
        e = UB == 16 ? launch_bwd_persist_t<T, 16, 32, 2>(a, nwg, lds, st)
                     : launch_bwd_persist_t<T, 8, 32, 2>(a, nwg, lds, st);
    } else if (per_wave <= 4) {
        e = UB == 16 ? launch_bwd_persist_t<T, 16, 32, 4>(a, nwg, lds, st)
                     : launch_bwd_persist_t<T, 8, 32, 4>(a, nwg, lds, st);
    } else {
        e = UB == 16 ? launch_bwd_persist_t<T, 16, 32, 6>(a, nwg, lds, st)
                     : launch_bwd_persist_t<T, 8, 32, 6>(a, nwg, lds, st);
    }
    if (timer_on && e == hipSuccess) (void)hipEventRecord(e1, st);
    return e;
}

template hipError_t launch_bwd_persist<float>(PBwdArgs&, hipStream_t, int, hipEvent_t, hipEvent_t);
template hipError_t launch_bwd_persist<bf16>(PBwdArgs&, hipStream_t, int, hipEvent_t, hipEvent_t);

// The large-batch backward (bf16, one direction per launch): returns an
// error before anything is enqueued when the grid does not fit the device.
hipError_t launch_bwd_big(PBwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1) {
    if (a.nslots != 1) return hipErrorInvalidValue;
    a.ntiles = (a.H + BB_UT - 1) / BB_UT;
    a.mgroups = (a.B + BB_MG - 1) / BB_MG;
    a.ngu = (a.H + BB_UG - 1) / BB_UG;
    a.ngk = (4 * a.H + BB_KG - 1) / BB_KG;
    const int nA = a.ntiles * a.mgroups, nB = a.mgroups * a.ngu * a.ngk;
    const int nwg = nA > nB ? nA : nB;
    const size_t lds = (size_t)4 * BB_MG * BB_RP * sizeof(float);
    hipError_t e = resident_limit((const void*)k_bwd_big, 64 * BB_NW, lds, nwg);
    if (e != hipSuccess) return e;
    if (timer_on) (void)hipEventRecord(e0, st);
    hipLaunchKernelGGL(k_bwd_big, dim3(nwg), dim3(64 * BB_NW), lds, st, a);
    e = hipGetLastError();
    if (timer_on && e == hipSuccess) (void)hipEventRecord(e1, st);
    return e;
}

}  // namespace lsd
