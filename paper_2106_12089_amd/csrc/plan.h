// Host-side layout of the mask, reserve and workspace buffers.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/lstm_sd.h"

namespace lsd {

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Plan {
    int L, I, H, B, T, D, dtype, compact;
    double p_nr[16], p_rh[16];   // per layer
    float s_nr[16], s_rh[16];    // 1/(1-p) computed in double, rounded to float
    int esize;            // bytes per element of x/W/U/h copies
    int G;                // 4H
    int BP;               // batch rounded up to 32 (transposed copies)
    int MGc;              // number of 64-row groups of the batch
    int sites, kmax, kin_max;
    int HP;               // H rounded up to 8 (row pitch of the per-step h buffer)
    int mtiles;           // 16-row tiles of the batch
    size_t das, hxs;      // elements of one fragment-major DA block / h exchange slot
    size_t xxs;           // elements of one layer-input exchange slot (stacked forward)

    // mask buffer
    size_t m_mask, m_keep, m_pos, m_count, m_drop, m_dcount, m_kseg, m_dseg, m_total;

    // reserve
    size_t r_gates, r_c, r_hrecT, r_dir_bytes;  // inside one (l, d) block
    size_t r_xT, r_h0T;                         // layer-0 input and h0, transposed
    size_t r_ybuf_base, r_ybuf_bytes;           // per layer l < L-1: ybuf then ybufT
    size_t r_ybufT_off;                         // offset of ybufT inside a layer block
    size_t r_total;

    // workspace
    size_t w_gx, w_hrec, w_hx, w_xx, w_gxs;     // forward (w_gxs: input products of the stacked layers above the first)
    size_t w_da, w_daT, w_dxw, w_dc, w_dhc, w_dxc;  // backward
    size_t w_part;                              // backward, large batch: [ceil(4H/512)][B][H] partial sums
    size_t w_sync;                              // barrier counters and error flag
    size_t w_loss, w_total;

    int kin(int l) const { return l == 0 ? I : D * H; }
    int site_nr(int l) const { return l; }
    int site_rh(int l, int d) const { return L + l * D + d; }
    int site_k(int s) const { return s < L ? kin(s) : H; }
    double site_p(int s) const { return s < L ? p_nr[s] : p_rh[(s - L) / D]; }
    int stream_id(int s) const {
        if (s < L) return 4 * s;
        int r = s - L, l = r / D, d = r % D;
        return 4 * l + 2 + d;
    }
    size_t rdir(int l, int d) const { return (size_t)(l * D + d) * r_dir_bytes; }
    size_t rybuf(int l) const { return r_ybuf_base + (size_t)l * r_ybuf_bytes; }
    size_t rybufT(int l) const { return rybuf(l) + r_ybufT_off; }
};

// Returns 0 and fills `p`, or a negative LSTM_SD_* code with a message.
int make_plan(const lstm_sd_dims* d, Plan* p, const char** why);

}  // namespace lsd
