// Kernel argument blocks and launchers shared by the host driver.
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
    int T, kmax, compact, generate;
    uint64_t seed, step;
    int K[MAX_SITES];
    int sid[MAX_SITES];
    uint64_t thr[MAX_SITES];
};

// Mask rows of one site: row t starts at +t*kmax (mask, keep, pos), count[t].
struct SiteView {
    const uint8_t* mask;
    const int32_t* keep;
    const int32_t* pos;
    const int32_t* count;
    int kmax;
};

// Gathered-K forward product of one layer/direction, all t in one launch:
//   Gx[t][b][n] = s * sum_{j < count_t} X[t][b][keep_t[j]] * W[keep_t[j]][n] + bias[n]
struct FxArgs {
    const void* X;  int ldx;            // X + (t*B + b)*ldx
    const void* W;                      // [K][N]
    const float* bias;
    SiteView site;
    float* Gx;                          // [T][B][N]
    int B, N, T;
    float s;
};

// One recurrent forward step, per direction (grid.z = direction).
struct StepDir {
    const void* hprev;                  // [B][H] rows of h_{prev} (dtype)
    const void* U;                      // [H][4H]
    const float* gx;                    // [B][4H] for this t
    const uint8_t* mask;                // RH site row at t
    const int32_t* keep;
    const int32_t* count;               // points at count_t
    float* gates;                       // [B][4H]
    float* cres;                        // [B][H]
    void* hrec;                         // [B][H] dtype
    float* hT;                          // [B][H] fp32 state, in place
    float* cT;                          // [B][H] fp32 state, in place
    float* y;                           // top layer output rows + d*H, or null
    void* ybuf;                         // inter-layer output rows + d*H, or null
    int t;
};
struct StepArgs {
    StepDir d[2];
    const int32_t* lengths;
    int B, H, ldy;
    float s;
};

// Backward pointwise of one step (Eq. 7-9 and the activation derivatives).
struct BwdPwDir {
    const float* gates;                 // [B][4H] at t
    const float* cres;                  // c_t [B][H]
    const float* cprev;                 // c_{prev} [B][H] (reserve or c0)
    const float* dy;                    // full rows + d*H (top layer), or null
    const float* dxc;                   // compacted rows of the layer above, or null
    const int32_t* dxpos;               // NR pos row of the layer above at t (offset by d*H)
    const float* dhrec;                 // compacted recurrent gradient, or null
    const int32_t* rhpos;               // RH pos row of the step it came from
    float* dhc;                         // [B][H] pass-through carry, in place
    float* dcs;                         // [B][H] cell gradient carry, in place
    void* da;                           // [B][4H] dtype
    float* dbpart;                      // [4H] for this t
    int t;
};
struct BwdPwArgs {
    BwdPwDir d[2];
    const int32_t* lengths;
    int B, H, ldy, lddx;
};

// Gathered-N backward product: out[b][j] = s * m * sum_n DA[b][n] * Wt[keep[j]][n]
// (for the recurrent step: one t, grid.z = direction; for dX: grid.z = t and
// the directions are summed).
struct DhDir {
    const void* da;                     // [B][G] rows (dtype)
    const void* Wk;                     // [K][G] weight with the gathered rows
    const uint8_t* mask;
    const int32_t* keep;
    const int32_t* count;
    float* out;                         // [B][ldo] compacted output
};
struct DhArgs {
    DhDir d[2];
    int B, G, ldo;
    float s;
};

struct DxArgs {
    const void* da[2];                  // DA_d base [T][B][G]
    const void* W[2];                   // [K][G]
    SiteView site;
    float* out;                         // [T][B][ldo]
    int D, B, G, ldo, T;
    float s;
};

// Row-scatter weight gradient of one layer/direction:
//   dW[keep_t[j]][n] += s * sum_b act_t[b][keep_t[j]] * DA[t][b][n]
struct WgArgs {
    const void* act;                    // activations: act + t*act_tstride, rows ld act_ld
    long act_tstride; int act_ld;
    const void* act_first;              // if non-null, replaces act at t == t_first
    int t_first; int act_shift;         // act index for t is t + act_shift (h_prev indexing)
    const void* da;                     // [T][B][G]
    SiteView site;
    float* dW;                          // [K][G]
    int K, B, G, T;
    float s;
};

// Final step of a layer's backward pass.
struct FinalDir {
    const float* dhrec; const int32_t* rhpos; const float* dhc; const float* dcs;
    float* dh0; float* dc0;
};
struct FinalArgs { FinalDir d[2]; int B, H; };

}  // namespace lsd
