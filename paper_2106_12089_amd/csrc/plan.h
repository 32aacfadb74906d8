// Host-side layout of the mask, reserve and workspace buffers.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/lstm_sd.h"

namespace lsd {

inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Plan {
    int L, I, H, B, T, D, dtype, compact;
    double p_nr, p_rh;
    float s_nr, s_rh;     // 1/(1-p) computed in double, rounded to float
    int esize;            // bytes per element of x/W/U/h copies
    int G;                // 4H
    int sites, kmax, kin_max;

    // mask buffer
    size_t m_mask, m_keep, m_pos, m_count, m_total;

    // reserve: per (l, d) block, then per-layer inter-layer outputs
    size_t r_gates, r_c, r_hrec, r_dir_bytes;   // offsets inside one (l,d) block
    size_t r_ybuf_base, r_ybuf_bytes;           // ybuf for layers 0..L-2
    size_t r_total;

    // workspace
    size_t w_gx;                                // forward: D x [T][B][4H] f32
    size_t w_da, w_dbpart, w_dhrec, w_dc, w_dhc, w_dxc, w_bwd_end;
    size_t w_loss;                              // last 16 KiB: loss partials
    size_t w_total;

    int kin(int l) const { return l == 0 ? I : D * H; }
    int site_nr(int l) const { return l; }
    int site_rh(int l, int d) const { return L + l * D + d; }
    int site_k(int s) const { return s < L ? kin(s) : H; }
    int stream_id(int s) const {
        if (s < L) return 4 * s;
        int r = s - L, l = r / D, d = r % D;
        return 4 * l + 2 + d;
    }

    // mask buffer accessors (byte offsets)
    size_t mask_at(int s, int t) const { return m_mask + ((size_t)s * T + t) * kmax; }
    size_t keep_at(int s, int t) const { return m_keep + ((size_t)s * T + t) * kmax * 4; }
    size_t pos_at(int s, int t) const { return m_pos + ((size_t)s * T + t) * kmax * 4; }
    size_t count_at(int s) const { return m_count + (size_t)s * T * 4; }

    size_t rdir(int l, int d) const { return (size_t)(l * D + d) * r_dir_bytes; }
    size_t rybuf(int l) const { return r_ybuf_base + (size_t)l * r_ybuf_bytes; }
};

// Returns 0 and fills `p`, or a negative LSTM_SD_* code with a message.
int make_plan(const lstm_sd_dims* d, Plan* p, const char** why);

}  // namespace lsd
