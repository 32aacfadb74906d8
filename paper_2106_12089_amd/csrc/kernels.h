// Kernel argument blocks shared by the host driver and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsd {

constexpr int MAX_SITES = 48;       // L <= 16 layers, D <= 2

struct MaskArgs {
    uint8_t* mask;
    int32_t* keep;
    int32_t* pos;
    int32_t* count;
    int32_t* drop;
    int32_t* dcount;
    int32_t* kseg;
    int32_t* dseg;
    int T, kmax, compact, generate;
    int fixed;                          // 1: every t takes the draw of t = 0 (one mask for the whole sequence)
    uint64_t seed, step;
    int K[MAX_SITES];
    int sid[MAX_SITES];
    uint64_t thr[MAX_SITES];
};

// Mask rows of one site: row t starts at +t*kmax (mask, keep, pos, drop),
// count[t], dcount[t].
struct SiteView {
    const uint8_t* mask;
    const int32_t* keep;
    const int32_t* pos;
    const int32_t* count;
    const int32_t* drop;
    const int32_t* dcount;
    const int32_t* kseg;                // [T][17]: keep-list offsets of 16 neuron segments
    const int32_t* dseg;                // [T][17]
    int kmax;
};

// src [N][B][K] -> dst [N][K][BP] (BP >= B; rows b >= B written as zero)
struct TransArgs {
    const void* src;
    void* dst;
    int B, K, BP;
    int n1;                             // matrices of the first job; the rest come from the second
    const void* src2;                   // second job (K2 columns), or unused when every matrix is the first job's
    void* dst2;
    int K2;
    // with n_init > 0, one more grid slice initialises the forward pass:
    // hT <- h0 (as float), cT <- c0 (n_init elements), barrier counters <- 0
    const void* h0;
    const float* c0;
    float *hT, *cT;
    long n_init;
    unsigned* bar;
    int* err;                           // (the status word follows at SYNC_STATUS_OFS - SYNC_ERR_OFS bytes)
};

// Forward input product of one layer/direction, all t in one launch:
//   Gx[t][b][n] = s * sum_{j < count_t} X[t][b][keep_t[j]] W[keep_t[j]][n] + bias[n]
struct FxArgs {
    const void* X; int ldx;             // X + (t*B + b)*ldx
    const void* W;                      // [K][G]
    int K;
    const float* bias;
    SiteView site;
    float* Gx;                          // [T][B][G]
    int B, G, T, dense;
    float s;
    // the input transposed, XT + t*xt_tstride + k*xt_ld + b, bf16: when set
    // (batch >= 64), the large-batch kernel runs (after the transposes)
    const void* XT; long xt_tstride; int xt_ld;
    // with tr_gz > 0, the launch also runs the transposes (and the pass
    // initialisation) of tr, as a virtual (tr_gx, tr_gy, tr_gz) grid of
    // workgroups past y = T; trN = its matrix count
    TransArgs tr;
    int trN, tr_gx, tr_gy, tr_gz;
};

// One recurrent forward step, per direction (grid.z = direction).
struct StepDir {
    const void* hprev;                  // [B][H] row-major h_prev (dtype)
    const void* U;                      // [H][4H]
    const float* gx;                    // [B][4H] at t
    const uint8_t* mask;                // RH site row at t
    const int32_t* keep;
    const int32_t* count;               // -> count_t
    float* gates;                       // [B][H][4] (the four gates of a unit together)
    float* cres;                        // [B][H]
    void* hrec;                         // [B][H] row-major h_t (dtype)
    void* hrecT;                        // [H][BP] h_t transposed (dtype)
    float* hT;                          // [B][H] fp32 state, in place
    float* cT;                          // [B][H] fp32 state, in place
    float* y;                           // top layer output rows + d*H, or null
    void* ybuf;                         // inter-layer output rows + d*H (ld ldy), or null
    void* ybufT;                        // inter-layer output transposed rows + d*H (ld BP), or null
    int t;
};
struct StepArgs {
    StepDir d[2];
    const int32_t* lengths;
    int B, H, ldy, BP, dense;
    float s;
};

// One backward step of BPTT for one direction: the output-sparse recurrent
// gradient of the step processed before (Eq. 10) for the kept units, then
// the pointwise backward (Eq. 7-9 and activation derivatives) at t.
struct BwdDir {
    // recurrent gradient from the previously processed step (has_next)
    const void* da_next;                // DA of that step, fragment-major [B][G] (dtype)
    const uint8_t* nmask;               // RH mask row of that step
    const int32_t* nkeep;               // kept units of that step
    const int32_t* ncount;
    const int32_t* ndrop;               // dropped units of that step
    const int32_t* ndcount;
    const int32_t* nkseg;               // [17] segment offsets of nkeep (slice x: 2x .. 2x+2)
    const int32_t* ndseg;               // [17] segment offsets of ndrop
    const void* U;                      // [H][G]
    // pointwise at t
    const float* gates;                 // [B][H][4]
    const float* cres;                  // c_t [B][H]
    const float* cprev;                 // c_prev [B][H]
    const float* dy;                    // top layer: rows + d*H (ld ldy), or null
    const float* dxc;                   // layer above: compacted rows (ld lddx), or null
    const int32_t* dxpos;               // NR pos row of the layer above at t, + d*H
    float* dhc;                         // [B][H] pass-through carry, in place
    float* dcs;                         // [B][H] cell-gradient carry, in place
    void* da;                           // DA_t, fragment-major [B][G] (dtype)
    void* daT;                          // [G][BP] dtype (transposed)
    float* dh0;                         // final pass: [B][H]
    float* dc0;
    int t;
};
struct BwdArgs {
    BwdDir d[2];
    const int32_t* lengths;
    int B, H, BP, ldy, lddx, tps, has_next, final_pass, dense;   // tps: tiles per XCD slice
    int mtiles;                         // 16-row tiles of the batch (fragment-major DA)
    float s;
};

// Output-sparse input gradient, all t, summed over directions:
//   out[t][b][j] = s * m * sum_d sum_n DA_d[t][b][n] W_d[keep_t[j]][n]
struct DxArgs {
    const void* da[2];                  // DA_d [T] x fragment-major [B][G]
    const void* W[2];                   // [K][G]
    SiteView site;
    float* out;                         // [T][B][ldo]: kept columns at their compact positions, or
    int scatter;                        //   (scatter) every column at its own, the dropped ones as zeros
    int D, B, G, ldo, T, K, tps, dense, mtiles;
    float s;
    const int* status;                  // sticky barrier status of the step, or null: when set, NaN is written
    int big;                            // bf16, batch >= 64: the large-batch kernel
};

// Weight gradient of one (layer, direction, site), summed over every step:
//   dW[k][n] = s * sum_t sum_b actT_t[k][b] DAT_t[n][b]
// over the rows k kept at t (row-sparse), or every row (times the mask byte
// in dense mode); rows never kept are 0.  dW (and db) are overwritten.
struct WgArgs {
    const void* actT;                   // actT + (t + shift)*tstride: [K][BP]
    long tstride;
    const void* actT_first;             // replaces actT at t == t_first (if non-null)
    int t_first, shift;
    const void* daT;                    // [T][G][BP]
    SiteView site;
    float* out;                         // dW [K][G]
    float* db;                          // non-null: also the bias gradient (Eq. 11), the sum of DA^T
    int K, B, BP, G, T, dense;
    int full;                           // every keep list of the site is the identity (p = 0, or dense mode)
    int staged;                         // (set at launch) a kernel with LDS-staged operands
    int fullmask;                       // (set at launch) a row-sparse problem on the full kernel, rows times the mask
    float s;
};
// Weight gradients of a pass (row-sparse and full problems) in one launch
constexpr int WG_MAXP = 8;
struct WgBatch {
    WgArgs p[WG_MAXP];
    int np;
    int big;                            // bf16 at a large batch: the register-accumulated kernel
    const int* status;                  // sticky barrier status of the step, or null: when set, NaN is written
};

// Persistent forward recurrence of one layer (both directions): one
// launch runs all T steps.
struct PFwdDir {
    const void* h0;                     // [B][H] row-major h0 (dtype)
    const void* U;                      // [H][4H]
    const float* gx;                    // [T][B][4H] input product incl. bias
    const float* c0;                    // [B][H]
    SiteView rh;                        // RH site of (l, d)
    float* gates;                       // [T][B][H][4] (the four gates of a unit together)
    float* cres;                        // [T][B][H]
    void* hrecT;                        // [T][H][BP]
    void* hx;                           // [2] fragment-major slots: h_t compacted by the next step's keep list
    float* hT;                          // [B][H]
    float* cT;                          // [B][H]
    float* y;                           // top layer: y + d*H (rows ld ldy, t stride B*ldy), or null
    void* ybuf;                         // inner layer: ybuf + d*H, or null
    void* ybufT;                        // inner layer: ybufT + d*H*BP (t stride ldy*BP), or null
    int dir;                            // 0: t = 0 .. T-1;  1: t = T-1 .. 0
    float s_rh, s_nr;                   // dropout scales of the slot's layer (RH; NR of its input)
    // A unidirectional stack whose layers run in one launch: each layer above
    // the first has an input-product worker slot, which forms
    // gx_t = s_nr * x~_t W + b (Eq. 1-4, input part) from x_t, the output of
    // the layer below that its slot publishes at step t; the layer reads gx
    // from the worker's output once the worker's counter covers step t.
    int role;                           // 0: a layer; 1: an input-product worker
    int dep;                            // worker: slot of the layer below; layer: slot of its worker; or -1
    const void* Win;                    // worker: [kin][4H]
    const float* bias;                  // worker: [4H]
    SiteView nr;                        // worker: NR site of the layer (keep lists of its input)
    const void* xin;                    // worker: [T] slots, fragment-major, compacted by nr
    int kin;                            // worker: input width
    float* gxo;                         // worker: [T][B][4H] output (the layer's gx)
    void* xout;                         // layer: [T] slots of its output for the layer above, or null
    SiteView nr_up;                     // layer: NR site of the layer above (compaction of xout)
};
// LDS row pitch of a transposed weight slice over K neurons: K rounded up to
// 32 (whole contraction chunks), plus 8 elements (16-byte rows that start on
// different banks)
__host__ __device__ inline int fwd_hp(int K) { return (K + 31) / 32 * 32 + 8; }

// Barrier counters of the persistent kernels: slot i has BAR_LINES counters
// (workgroup j adds to line j % BAR_LINES), line k at bar + BAR_PITCH *
// (BAR_LINES * i + k), a cache line each; the exit counter is line 0 of
// slot BAR_EXIT; the error flag sits at SYNC_ERR_OFS bytes.  The init kernel
// of a pass clears them, and each persistent launch leaves them clear for
// the next.
constexpr int BAR_PITCH = 64;
constexpr int BAR_LINES = 16;
static_assert((BAR_LINES & (BAR_LINES - 1)) == 0 && BAR_LINES <= 32, "counter lines: a power of 2, two slots per wave");
constexpr int BAR_EXIT = 8;
constexpr int SYNC_ERR_OFS = BAR_PITCH * 4 * (BAR_LINES * BAR_EXIT + 1);   // bytes
// Sticky status word (a cache line of its own): a persistent launch whose
// barrier wait timed out ORs its pass bit into it.  The forward pass's init
// clears it, nothing else does, so after a backward it tells whether the
// forward or the backward of that step failed; the weight- and
// input-gradient kernels read it and write NaN instead of values when set.
constexpr int SYNC_STATUS_OFS = SYNC_ERR_OFS + 128;
constexpr int STATUS_FWD = 1, STATUS_BWD = 2;
constexpr int SYNC_BYTES = SYNC_ERR_OFS + 256;

struct PFwdArgs {
    PFwdDir d[8];                       // slots: the directions of one layer, or the layers of a stack and their workers
    const int32_t* lengths;
    unsigned* bar;                      // barrier counters (BAR_LINES lines per slot; clear at launch)
    int* err;                           // barrier time-out flag
    long long timeout;                  // wall-clock ticks (<= 0: every wait fails at once)
    int B, H, HP, T, BP, ldy, dense, ntiles, mgroups, mtiles;
    int nslots, KP, kin_max;            // KP: LDS pitch of the W slices (0: no slot has Win)
    size_t wofs, kofs;                  // LDS offsets of the W slice and the keep lists (set by the launcher)
    size_t xxs;                         // elements per xin/xout slot
};

// Persistent BPTT of one layer (both directions): one launch
// runs all T backward steps and the final pass that forms dh0/dc0.
struct PBwdDir {
    const void* U;                      // [H][4H]
    SiteView rh;                        // RH site of (l, d)
    const float* gates;                 // [T][B][H][4]
    const float* cres;                  // [T][B][H]
    const float* c0;                    // [B][H]
    const float* dy;                    // top layer: dy + d*H (rows ld ldy, t stride B*ldy), or null
    const float* dxc;                   // inner layer: compacted dx of the layer above [T][B][lddx], or null
    const int32_t* dxpos;               // NR pos of the layer above, + d*H (t stride kmax)
    const float* dhT;                   // [B][H] or null
    const float* dcT;                   // [B][H] or null
    void* da;                           // [T] x fragment-major [B][4H] (exchange; also read by the dX product)
    void* daT;                          // [T][4H][BP]
    float* dh0;                         // [B][H]
    float* dc0;                         // [B][H]
    int dir;                            // 0: t = T-1 .. 0 (BP of the forward direction);  1: t = 0 .. T-1
    float s_rh, s_nr;                   // layer: its RH scale; worker: the NR scale of the layer above
    // A unidirectional stack in one launch: the input gradient of layer l+1
    // (Eq. 10, dx = s * da W^T over the kept inputs) is formed per step by a
    // worker slot from the DA layer l+1 publishes, and read by layer l.
    int role;                           // 0: the recurrence of one layer (direction); 1: input-gradient worker
    int src;                            // worker: slot of the layer whose DA it reads
    int above;                          // layer: worker slot that provides its dh input, or -1
    const float* dxw;                   // layer: [T][B][H] that input (with above)
    const void* Wup;                    // worker: input weights [H][4H] of the layer above
    SiteView nr_up;                     // worker: NR site of the layer above (output sparsity and scale)
    float* dxw_out;                     // worker: [T][B][H]
};
struct PBwdArgs {
    PBwdDir d[8];                       // slots: the directions of one layer, or the layers and workers of a stack
    const int32_t* lengths;
    unsigned* bar;
    int* err;
    long long timeout;                  // wall-clock ticks (<= 0: every wait fails at once)
    int B, H, T, BP, ldy, lddx, kmax, dense, ntiles, mgroups, mtiles, nslots;
    float* part;                        // large-batch kernel: [ngk][B][H] partial recurrent gradients
    int ngu, ngk;                       // large-batch kernel: unit groups and gate-column groups
};

}  // namespace lsd
