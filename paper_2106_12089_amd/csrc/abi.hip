// C ABI of the structured-dropout LSTM step: validation, buffer layout and
// the launch sequence of forward and backward.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <type_traits>
#include <mutex>
#include <string>

#include "../../include/lstm_sd.h"
#include "device.h"
#include "kernels.h"
#include "plan.h"

namespace lsd {

void launch_mask_build(const MaskArgs& a, int sites, hipStream_t st);
template <typename T> void launch_fx(const FxArgs& a, hipStream_t st);
template <typename T> void launch_step(const StepArgs& a, int D, hipStream_t st);
template <typename T> void launch_bwd(const BwdArgs& a, int D, hipStream_t st);
template <typename T> void launch_dx(const DxArgs& a, int K, hipStream_t st);
template <typename T> void launch_wgrad(const WgBatch& b, hipStream_t st);
void launch_bwd_init(const float*, const float*, float*, float*, long, void*, int, int, int, long, long, unsigned*, int*,
                     hipStream_t);
void launch_emb_grad(const int32_t*, int, int, int, const float*, const SiteView&, int, float*, hipStream_t);
void launch_case1_drop(int, int, const void*, void*, uint8_t*, int, int, int, uint64_t, uint64_t, uint64_t, uint64_t,
                       float, hipStream_t);
void launch_case1_undrop(const float*, const uint8_t*, float*, long, float, hipStream_t);
template <typename T> void launch_head_prep(const float*, void*, void*, int, int, int, int, hipStream_t);
void launch_ce_loss(const float*, const int32_t*, const int32_t*, int, int, int, float*, float*, float*, float*, float*,
                    hipStream_t);
template <typename T>
void launch_ce_grad(const float*, const int32_t*, const int32_t*, const float*, const float*, int, int, int, int, int,
                    void*, void*, hipStream_t);
void launch_mse(const float*, const float*, const int32_t*, float*, float*, int, float*, int, int, int,
                hipStream_t);
int setup_kernel_attributes();
bool timer_pair(int kid, hipEvent_t* e0, hipEvent_t* e1);
void timer_unpair();
template <typename T>
hipError_t launch_fwd_persist(PFwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1);
constexpr int KID_FWDP_ = 7;
constexpr int KID_BWDP_ = 8;
template <typename T>
hipError_t launch_bwd_persist(PBwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_fwd_big(PFwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_bwd_big(PBwdArgs& a, hipStream_t st, int timer_on, hipEvent_t e0, hipEvent_t e1);
bool wgrad_big_fits(int B);
int kernel_timer_start(const char* name);
int kernel_timer_stop(double* total_ms, int64_t* launches);

static thread_local std::string g_err;

static int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

static float inv_keep(double p) { return p > 0.0 ? (float)(1.0 / (1.0 - p)) : 1.0f; }

int make_plan(const lstm_sd_dims* d, Plan* p, const char** why) {
    if (!d) { *why = "dims is NULL"; return LSTM_SD_EINVAL; }
    if (d->num_layers < 1 || d->input_dim < 1 || d->hidden < 1 || d->batch < 1 || d->seq_len < 1) {
        *why = "dimensions must be >= 1"; return LSTM_SD_EINVAL;
    }
    if (d->num_dirs != 1 && d->num_dirs != 2) { *why = "num_dirs must be 1 or 2"; return LSTM_SD_EINVAL; }
    if (!(d->p_nr >= 0.0 && d->p_nr < 1.0) || !(d->p_rh >= 0.0 && d->p_rh < 1.0)) {
        *why = "dropout rates must be in [0, 1)"; return LSTM_SD_EINVAL;
    }
    for (int l = 0; l < d->num_layers && l < 16; ++l) {
        const double a = d->p_nr_layer ? d->p_nr_layer[l] : 0.0, b = d->p_rh_layer ? d->p_rh_layer[l] : 0.0;
        if (!(a >= 0.0 && a < 1.0) || !(b >= 0.0 && b < 1.0)) {
            *why = "per-layer dropout rates must be in [0, 1)"; return LSTM_SD_EINVAL;
        }
    }
    if (d->compact != 0 && d->compact != 1) { *why = "compact must be 0 or 1"; return LSTM_SD_EINVAL; }
    if (d->dtype != LSTM_SD_DTYPE_F32 && d->dtype != LSTM_SD_DTYPE_BF16) {
        *why = "dtype must be 0 (f32) or 1 (bf16)"; return LSTM_SD_EUNSUPPORTED;
    }
    if (d->num_layers > 16) { *why = "at most 16 layers"; return LSTM_SD_EUNSUPPORTED; }
    const long kin1 = (long)d->num_dirs * d->hidden;
    if (d->input_dim > LSTM_SD_MAX_K || kin1 > LSTM_SD_MAX_K || d->hidden > LSTM_SD_MAX_K) {
        *why = "input_dim, hidden and num_dirs*hidden must be <= LSTM_SD_MAX_K"; return LSTM_SD_EUNSUPPORTED;
    }
    if ((long)d->batch * d->seq_len > (1L << 24) || d->batch > 65536 || d->seq_len > 65535) {
        *why = "batch*seq_len too large"; return LSTM_SD_EUNSUPPORTED;
    }
    Plan& q = *p;
    q.L = d->num_layers; q.I = d->input_dim; q.H = d->hidden; q.B = d->batch; q.T = d->seq_len;
    q.D = d->num_dirs; q.dtype = d->dtype; q.compact = d->compact;
    for (int l = 0; l < 16; ++l) {
        const bool in = l < q.L;
        q.p_nr[l] = in && d->p_nr_layer ? d->p_nr_layer[l] : d->p_nr;
        q.p_rh[l] = in && d->p_rh_layer ? d->p_rh_layer[l] : d->p_rh;
        q.s_nr[l] = inv_keep(q.p_nr[l]);
        q.s_rh[l] = inv_keep(q.p_rh[l]);
    }
    q.esize = d->dtype == LSTM_SD_DTYPE_BF16 ? 2 : 4;
    q.G = 4 * q.H;
    q.BP = (q.B + 31) / 32 * 32;
    q.HP = (q.H + 7) / 8 * 8;
    q.mtiles = (q.B + 15) / 16;
    q.das = (size_t)((q.G + 31) / 32) * q.mtiles * 512;   // DA block per step: fragment-major [B][4H]
    q.hxs = (size_t)((q.H + 31) / 32) * q.mtiles * 512;
    q.xxs = (size_t)((q.D * q.H + 31) / 32) * q.mtiles * 512;
    q.MGc = (q.B + 63) / 64;
    q.sites = q.L + q.L * q.D;
    q.kin_max = q.L > 1 ? (q.I > q.D * q.H ? q.I : q.D * q.H) : q.I;
    q.kmax = q.kin_max > q.H ? q.kin_max : q.H;

    const size_t A = 256, T = q.T, B = q.B, H = q.H, G = q.G, D = q.D, BP = q.BP, es = q.esize;
    const size_t S = q.sites, KM = q.kmax;
    size_t off = 0;
    q.m_mask = off;   off = align_up(off + S * T * KM, A);
    q.m_keep = off;   off = align_up(off + S * T * KM * 4, A);
    q.m_pos = off;    off = align_up(off + S * T * KM * 4, A);
    q.m_count = off;  off = align_up(off + S * T * 4, A);
    q.m_drop = off;   off = align_up(off + S * T * KM * 4, A);
    q.m_dcount = off; off = align_up(off + S * T * 4, A);
    q.m_kseg = off;   off = align_up(off + S * T * 17 * 4, A);
    q.m_dseg = off;   off = align_up(off + S * T * 17 * 4, A);
    q.m_total = off;

    off = 0;
    q.r_gates = off; off = align_up(off + T * B * G * 4, A);
    q.r_c = off;     off = align_up(off + T * B * H * 4, A);
    q.r_hrecT = off; off = align_up(off + T * H * BP * es, A);
    q.r_dir_bytes = off;
    off = (size_t)q.L * D * q.r_dir_bytes;
    q.r_xT = off;    off = align_up(off + T * (size_t)q.I * BP * es, A);
    q.r_h0T = off;   off = align_up(off + (size_t)q.L * D * H * BP * es, A);
    q.r_ybuf_base = off;
    q.r_ybufT_off = align_up(T * B * D * H * es, A);
    q.r_ybuf_bytes = q.r_ybufT_off + align_up(T * D * H * BP * es, A);
    q.r_total = q.r_ybuf_base + (size_t)(q.L - 1) * q.r_ybuf_bytes;

    off = 0;
    q.w_gx = off;   off = align_up(off + D * T * B * G * 4, A);
    q.w_hrec = off; off = align_up(off + D * 2 * B * (size_t)q.HP * es, A);
    q.w_hx = off;   off = align_up(off + (D > (size_t)q.L ? D : (size_t)q.L) * 2 * (size_t)q.hxs * es, A);
    q.w_xx = off;   off = align_up(off + (size_t)(q.L - 1) * T * q.xxs * es, A);
    q.w_gxs = off;  off = align_up(off + (q.D == 1 ? (size_t)(q.L - 1) * T * B * G * 4 : 0), A);
    const size_t fwd = off;
    off = 0;
    const size_t NR = D > (size_t)q.L ? D : (size_t)q.L;   // DA regions: per direction, or per layer of a stack
    q.w_da = off;     off = align_up(off + NR * T * (size_t)q.das * es, A);
    q.w_daT = off;    off = align_up(off + NR * T * G * BP * es, A);
    q.w_dxw = off;    off = align_up(off + (size_t)(q.L - 1) * T * B * H * 4, A);
    q.w_dc = off;     off = align_up(off + D * B * H * 4, A);
    q.w_dhc = off;    off = align_up(off + D * B * H * 4, A);
    q.w_dxc = off;    off = align_up(off + 2 * T * B * (size_t)q.kin_max * 4, A);
    q.w_part = off;   off = align_up(off + (size_t)((4 * q.H + 511) / 512) * B * H * 4, A);
    const size_t bwd = off;
    q.w_sync = align_up(fwd > bwd ? fwd : bwd, A);
    q.w_loss = q.w_sync + align_up(SYNC_BYTES, A);   // barrier counters and error flag
    q.w_total = q.w_loss + 16384;
    return LSTM_SD_OK;
}

// Persistent recurrent kernels are used unless LSTM_SD_PERSIST=0 (a debug
// switch that forces the per-step kernels).
// LSTM_SD_STACK=0 runs a unidirectional stack one layer per launch
static bool use_stacked() {
    const char* v = getenv("LSTM_SD_STACK");
    return !(v && v[0] == '0');
}

// LSTM_SD_FWD_WORKERS=0: a stacked forward without input-product workers
static bool use_fwd_workers() {
    const char* v = getenv("LSTM_SD_FWD_WORKERS");
    return !(v && v[0] == '0');
}

// The large-batch persistent kernels (bf16) run where the row-group tiling
// does not fit.  LSTM_SD_BIG=0: never (per-step kernels there instead);
// LSTM_SD_BIG=2: wherever they apply, one launch per layer (tests of their
// tiling on ragged shapes).
static int big_mode() {
    const char* v = getenv("LSTM_SD_BIG");
    return (v && v[0] == '0') ? 0 : (v && v[0] == '2') ? 2 : 1;
}
static bool use_big() { return big_mode() != 0; }
// LSTM_SD_WGRAD_BIG=0: the weight gradients of a large batch on the
// small-batch kernel
static bool use_wgrad_big() {
    const char* v = getenv("LSTM_SD_WGRAD_BIG");
    return !(v && v[0] == '0');
}

// LSTM_SD_GEMM_BIG=0: the input products and input gradients of a large
// batch on the small-batch kernels
static bool use_gemm_big() {
    const char* v = getenv("LSTM_SD_GEMM_BIG");
    return !(v && v[0] == '0');
}

static bool use_persistent() {
    const char* v = getenv("LSTM_SD_PERSIST");
    return !(v && v[0] == '0');
}

// Grid-barrier time-out of the persistent kernels: 0.5 s by default, or
// what lstm_sd_set_barrier_timeout set (process-wide), in wall-clock ticks.
static std::atomic<double> g_timeout_s{-1.0};
static long long barrier_timeout_ticks() {
    static int khz = 0;
    if (!khz) {
        int dev = 0, k = 0;
        if (hipGetDevice(&dev) != hipSuccess) dev = 0;
        if (hipDeviceGetAttribute(&k, hipDeviceAttributeWallClockRate, dev) != hipSuccess || k <= 0) k = 100000;
        khz = k;
    }
    const double sec = g_timeout_s.load();
    if (sec < 0.0) return (long long)khz * 500;
    return (long long)(sec * 1000.0 * khz);
}

static int hip_check(const char* where) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(LSTM_SD_EHIP, std::string(where) + ": " + hipGetErrorString(e));
    return LSTM_SD_OK;
}

static SiteView site_view(const Plan& P, const void* mbuf, int s) {
    const char* m = (const char*)mbuf;
    const size_t row = (size_t)s * P.T * P.kmax;
    SiteView v;
    v.mask = (const uint8_t*)(m + P.m_mask) + row;
    v.keep = (const int32_t*)(m + P.m_keep) + row;
    v.pos = (const int32_t*)(m + P.m_pos) + row;
    v.count = (const int32_t*)(m + P.m_count) + (size_t)s * P.T;
    v.drop = (const int32_t*)(m + P.m_drop) + row;
    v.dcount = (const int32_t*)(m + P.m_dcount) + (size_t)s * P.T;
    v.kseg = (const int32_t*)(m + P.m_kseg) + (size_t)s * P.T * 17;
    v.dseg = (const int32_t*)(m + P.m_dseg) + (size_t)s * P.T * 17;
    v.kmax = P.kmax;
    return v;
}

static uint64_t threshold64(double p) {
    // floor(p * 2^64), exact: p = mant * 2^(e-53) with a 53-bit integer mantissa
    if (p <= 0.0) return 0;
    int e;
    const double m = frexp(p, &e);                 // p = m * 2^e, 0.5 <= m < 1
    const uint64_t mant = (uint64_t)ldexp(m, 53);  // exact
    const int sh = e + 64 - 53;                    // p * 2^64 = mant * 2^sh
    if (sh >= 0) return sh >= 64 ? 0 : (mant << sh);
    return -sh >= 64 ? 0 : (mant >> (-sh));
}

static int do_masks(const lstm_sd_dims* dims, uint64_t seed, uint64_t step, void* mbuf, size_t mbytes,
                    void* stream, int generate, int fixed = 0) {
    Plan P;
    const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!mbuf) return fail(LSTM_SD_EINVAL, "mask_buf is NULL");
    if (mbytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_mask_bytes()");
    MaskArgs a;
    memset(&a, 0, sizeof(a));
    char* m = (char*)mbuf;
    a.mask = (uint8_t*)(m + P.m_mask);
    a.keep = (int32_t*)(m + P.m_keep);
    a.pos = (int32_t*)(m + P.m_pos);
    a.count = (int32_t*)(m + P.m_count);
    a.drop = (int32_t*)(m + P.m_drop);
    a.dcount = (int32_t*)(m + P.m_dcount);
    a.kseg = (int32_t*)(m + P.m_kseg);
    a.dseg = (int32_t*)(m + P.m_dseg);
    a.T = P.T; a.kmax = P.kmax; a.compact = P.compact; a.generate = generate; a.fixed = fixed;
    a.seed = seed; a.step = step;
    for (int s = 0; s < P.sites; ++s) {
        a.K[s] = P.site_k(s);
        a.sid[s] = P.stream_id(s);
        a.thr[s] = threshold64(P.site_p(s));
    }
    launch_mask_build(a, P.sites, (hipStream_t)stream);
    return hip_check("mask kernel launch");
}

template <typename E>
static int forward_impl(const Plan& P, const lstm_sd_weights* w, const void* x, const int32_t* lengths,
                        const void* h0, const float* c0, const void* mbuf, float* y, float* hT, float* cT,
                        void* reserve, void* ws, hipStream_t st) {
    const int L = P.L, D = P.D, T = P.T, B = P.B, H = P.H, G = P.G, BP = P.BP;
    const size_t es = P.esize;
    char* R = (char*)reserve;
    char* W = (char*)ws;
    // x (T matrices) and h0 (L*D matrices) transposed, and the pass
    // initialised (hT, cT, barrier counters): these ride on the first input
    // product launch (independent work, one launch less)
    TransArgs tr;
    memset(&tr, 0, sizeof(tr));
    tr.src = x; tr.dst = R + P.r_xT; tr.B = B; tr.K = P.I; tr.BP = BP; tr.n1 = T;
    tr.src2 = h0; tr.dst2 = R + P.r_h0T; tr.K2 = H;
    tr.h0 = h0; tr.c0 = c0; tr.hT = hT; tr.cT = cT; tr.n_init = (long)L * D * B * H;
    tr.bar = (unsigned*)(W + P.w_sync); tr.err = (int*)(W + P.w_sync + SYNC_ERR_OFS);
    bool tr_pending = true;
    // large batches (bf16): the input products read the transposed inputs
    const bool gemm_big = std::is_same<E, bf16>::value && B >= 64 && use_gemm_big();
    auto attach_tr = [&](FxArgs& f) {
        if (!tr_pending) return;
        f.tr = tr;
        f.trN = T + L * D;
        f.tr_gx = ((P.I > H ? P.I : H) + 31) / 32;
        f.tr_gy = BP / 32;
        f.tr_gz = T + L * D + 1;
        tr_pending = false;
    };
    // Unidirectional stack: every layer's recurrence in one persistent
    // launch, layer l one step behind layer l-1, each layer above the first
    // computing its input product from what the layer below published.
    auto fill_slot = [&](PFwdDir& pd, int l, int d) {
        const int k = l * D + d;
        char* rd = R + P.rdir(l, d);
        pd.h0 = (const char*)h0 + (size_t)k * B * H * es;
        pd.U = w->U[k];
        pd.gx = (const float*)(W + P.w_gx) + (size_t)d * T * B * G;
        pd.c0 = c0 + (size_t)k * B * H;
        pd.rh = site_view(P, mbuf, P.site_rh(l, d));
        pd.gates = (float*)(rd + P.r_gates);
        pd.cres = (float*)(rd + P.r_c);
        pd.hrecT = rd + P.r_hrecT;
        pd.hT = hT + (size_t)k * B * H;
        pd.cT = cT + (size_t)k * B * H;
        pd.dir = d;
        pd.s_rh = P.s_rh[l];
        pd.s_nr = P.s_nr[l];
        pd.role = 0;
        pd.dep = -1;
        if (l == L - 1) {
            pd.y = y + d * H;
        } else {
            pd.ybuf = R + P.rybuf(l) + (size_t)d * H * es;
            pd.ybufT = R + P.rybufT(l) + (size_t)d * H * BP * es;
        }
    };
    auto common_args = [&](PFwdArgs& pa) {
        memset(&pa, 0, sizeof(pa));
        pa.lengths = lengths;
        pa.bar = (unsigned*)(W + P.w_sync);
        pa.err = (int*)(W + P.w_sync + SYNC_ERR_OFS);
        pa.timeout = barrier_timeout_ticks();
        pa.B = B; pa.H = H; pa.HP = P.HP; pa.T = T; pa.BP = BP; pa.ldy = D * H; pa.dense = !P.compact;
        pa.mtiles = P.mtiles;
        pa.xxs = P.xxs;
    };
    auto launch_fx_layer = [&](int l) {
        const int kin = P.kin(l);
        const void* X = l == 0 ? x : (const void*)(R + P.rybuf(l - 1));
        for (int d = 0; d < D; ++d) {
            FxArgs f;
            memset(&f, 0, sizeof(f));
            f.X = X; f.ldx = kin;
            f.W = w->W[l * D + d];
            f.bias = w->b[l * D + d];
            f.site = site_view(P, mbuf, P.site_nr(l));
            f.Gx = (float*)(W + P.w_gx) + (size_t)d * T * B * G;
            f.K = kin; f.B = B; f.G = G; f.T = T; f.dense = !P.compact; f.s = P.s_nr[l];
            if (gemm_big) {
                f.XT = l == 0 ? (const void*)(R + P.r_xT) : (const void*)(R + P.rybufT(l - 1));
                f.xt_tstride = (long)kin * BP;
                f.xt_ld = BP;
            }
            attach_tr(f);
            launch_fx<E>(f, st);
        }
    };
    // A unidirectional stack in one launch: with an input-product worker
    // slot per layer above the first (slots: layer 0, then worker l at 2l-1
    // and layer l at 2l), or, when that grid does not fit, with each layer
    // forming its own input product (slot l).
    auto stacked = [&](bool workers) -> bool {
        PFwdArgs pa;
        common_args(pa);
        pa.nslots = workers ? 2 * L - 1 : L;
        pa.kin_max = P.kin(1);
        pa.KP = fwd_hp(pa.kin_max);
        for (int l = 0; l < L; ++l) {
            const int sl = workers && l > 0 ? 2 * l : l;
            PFwdDir& pd = pa.d[sl];
            fill_slot(pd, l, 0);
            pd.hx = W + P.w_hx + (size_t)l * 2 * P.hxs * es;
            if (l > 0) {
                PFwdDir& xs = workers ? pa.d[sl - 1] : pd;      // the slot forming the input product
                if (workers) {
                    fill_slot(xs, l, 0);
                    xs.role = 1;
                    xs.gxo = (float*)(W + P.w_gxs) + (size_t)(l - 1) * T * B * G;
                    pd.gx = xs.gxo;
                    pd.dep = sl - 1;
                }
                xs.dep = workers ? sl - 2 : l - 1;              // the layer below
                xs.Win = w->W[l];
                xs.bias = w->b[l];
                xs.nr = site_view(P, mbuf, P.site_nr(l));
                xs.xin = W + P.w_xx + (size_t)(l - 1) * T * P.xxs * es;
                xs.kin = P.kin(l);
            }
            if (l < L - 1) {
                pd.xout = W + P.w_xx + (size_t)l * T * P.xxs * es;
                pd.nr_up = site_view(P, mbuf, P.site_nr(l + 1));
            }
        }
        hipEvent_t e0 = nullptr, e1 = nullptr;
        const bool timed = timer_pair(KID_FWDP_, &e0, &e1);
        if (launch_fwd_persist<E>(pa, st, timed, e0, e1) == hipSuccess) return true;
        (void)hipGetLastError();              // does not fit
        if (timed) timer_unpair();
        return false;
    };
    const bool big_first = std::is_same<E, bf16>::value && big_mode() == 2;
    bool fx0_done = false;
    if (use_persistent() && use_stacked() && !big_first && D == 1 && L > 1 && L <= 4) {
        launch_fx_layer(0);
        if ((use_fwd_workers() && stacked(true)) || stacked(false)) return hip_check("forward launch");
        fx0_done = true;                      // neither fits: one layer at a time below
    }
    for (int l = 0; l < L; ++l) {
        const int kin = P.kin(l);
        const void* X = l == 0 ? x : (const void*)(R + P.rybuf(l - 1));
        for (int d = 0; d < D && !(l == 0 && fx0_done); ++d) {
            FxArgs f;
            memset(&f, 0, sizeof(f));
            f.X = X; f.ldx = kin;
            f.W = w->W[l * D + d];
            f.bias = w->b[l * D + d];
            f.site = site_view(P, mbuf, P.site_nr(l));
            f.Gx = (float*)(W + P.w_gx) + (size_t)d * T * B * G;
            f.K = kin; f.B = B; f.G = G; f.T = T; f.dense = !P.compact; f.s = P.s_nr[l];
            if (gemm_big) {
                f.XT = l == 0 ? (const void*)(R + P.r_xT) : (const void*)(R + P.rybufT(l - 1));
                f.xt_tstride = (long)kin * BP;
                f.xt_ld = BP;
            }
            attach_tr(f);
            launch_fx<E>(f, st);
        }
        if (use_persistent()) {
            PFwdArgs pa;
            common_args(pa);
            pa.nslots = D;
            for (int d = 0; d < D; ++d) {
                fill_slot(pa.d[d], l, d);
                pa.d[d].hx = W + P.w_hx + (size_t)d * 2 * P.hxs * es;
            }
            hipEvent_t e0 = nullptr, e1 = nullptr;
            const bool timed = timer_pair(KID_FWDP_, &e0, &e1);
            if (big_first && launch_fwd_big(pa, st, timed, e0, e1) == hipSuccess) continue;
            (void)hipGetLastError();
            if (launch_fwd_persist<E>(pa, st, timed, e0, e1) == hipSuccess) continue;
            (void)hipGetLastError();          // does not fit: the large-batch kernel (bf16), else per step
            if (std::is_same<E, bf16>::value && use_big() && launch_fwd_big(pa, st, timed, e0, e1) == hipSuccess)
                continue;
            (void)hipGetLastError();
            if (timed) timer_unpair();
        }
        for (int s = 0; s < T; ++s) {
            StepArgs a;
            memset(&a, 0, sizeof(a));
            a.lengths = lengths; a.B = B; a.H = H; a.ldy = D * H; a.BP = BP; a.dense = !P.compact; a.s = P.s_rh[l];
            for (int d = 0; d < D; ++d) {
                const int k = l * D + d;
                const int t = d == 0 ? s : T - 1 - s;
                char* rd = R + P.rdir(l, d);
                char* hrec2 = W + P.w_hrec + (size_t)d * 2 * B * P.HP * es;
                StepDir& sd = a.d[d];
                sd.t = t;
                sd.hprev = s == 0 ? (const void*)((const char*)h0 + (size_t)k * B * H * es)
                                  : (const void*)(hrec2 + (size_t)((s - 1) & 1) * B * P.HP * es);
                sd.hrec = hrec2 + (size_t)(s & 1) * B * P.HP * es;
                sd.hrecT = rd + P.r_hrecT + (size_t)t * H * BP * es;
                sd.U = w->U[k];
                sd.gx = (const float*)(W + P.w_gx) + ((size_t)d * T + t) * B * G;
                const SiteView sv = site_view(P, mbuf, P.site_rh(l, d));
                sd.mask = sv.mask + (size_t)t * P.kmax;
                sd.keep = sv.keep + (size_t)t * P.kmax;
                sd.count = sv.count + t;
                sd.gates = (float*)(rd + P.r_gates) + (size_t)t * B * G;
                sd.cres = (float*)(rd + P.r_c) + (size_t)t * B * H;
                sd.hT = hT + (size_t)k * B * H;
                sd.cT = cT + (size_t)k * B * H;
                if (l == L - 1) {
                    sd.y = y + (size_t)t * B * D * H + d * H;
                } else {
                    sd.ybuf = R + P.rybuf(l) + ((size_t)t * B * D * H + d * H) * es;
                    sd.ybufT = R + P.rybufT(l) + ((size_t)t * D * H + d * H) * BP * es;
                }
            }
            launch_step<E>(a, D, st);
        }
    }
    return hip_check("forward launch");
}

template <typename E>
static int backward_impl(const Plan& P, const lstm_sd_weights* w, const int32_t* lengths,
                         const float* c0, const void* mbuf, const void* reserve,
                         const float* dy, const float* dhT, const float* dcT, float* dx, float* dh0,
                         float* dc0, const lstm_sd_grads* g, void* ws, hipStream_t st) {
    const int L = P.L, D = P.D, T = P.T, B = P.B, H = P.H, G = P.G, BP = P.BP;
    const size_t es = P.esize;
    const char* R = (const char*)reserve;
    char* W = (char*)ws;
    unsigned* sync_bar = (unsigned*)(W + P.w_sync);
    int* sync_err = (int*)(W + P.w_sync + SYNC_ERR_OFS);
    const int* sync_status = (const int*)(W + P.w_sync + SYNC_STATUS_OFS);
    const int tps_h = ((H + 7) / 8 + 15) / 16;     // 16-unit tiles per XCD slice of the hidden units
    // DA and DA^T regions: one per direction, or one per layer when a
    // unidirectional stack runs in one launch
    auto da_of = [&](int reg) { return W + P.w_da + (size_t)reg * T * P.das * es; };
    auto daT_of = [&](int reg) { return W + P.w_daT + (size_t)reg * T * G * BP * es; };
    auto common_args = [&](PBwdArgs& pa) {
        memset(&pa, 0, sizeof(pa));
        pa.lengths = lengths;
        pa.bar = (unsigned*)(W + P.w_sync);
        pa.err = (int*)(W + P.w_sync + SYNC_ERR_OFS);
        pa.timeout = barrier_timeout_ticks();
        pa.B = B; pa.H = H; pa.T = T; pa.BP = BP; pa.ldy = D * H;
        pa.kmax = P.kmax; pa.dense = !P.compact; pa.mtiles = P.mtiles;
    };
    auto fill_layer = [&](PBwdDir& pd, int l, int d, int reg) {
        const int k = l * D + d;
        const char* rd = R + P.rdir(l, d);
        pd.U = w->U[k];
        pd.rh = site_view(P, mbuf, P.site_rh(l, d));
        pd.gates = (const float*)(rd + P.r_gates);
        pd.cres = (const float*)(rd + P.r_c);
        pd.c0 = c0 + (size_t)k * B * H;
        if (l == L - 1) pd.dy = dy + d * H;
        pd.dhT = dhT ? dhT + (size_t)k * B * H : nullptr;
        pd.dcT = dcT ? dcT + (size_t)k * B * H : nullptr;
        pd.da = da_of(reg);
        pd.daT = daT_of(reg);
        pd.dh0 = dh0 + (size_t)k * B * H;
        pd.dc0 = dc0 + (size_t)k * B * H;
        pd.dir = d;
        pd.s_rh = P.s_rh[l];
        pd.above = -1;
    };
    // input gradient of layer l for the layer below (and the caller's dx)
    auto layer_dx = [&](int l, int reg0, float* dxc_here) {
        const int kin = P.kin(l);
        const SiteView nv = site_view(P, mbuf, P.site_nr(l));
        DxArgs a;
        memset(&a, 0, sizeof(a));
        for (int d = 0; d < D; ++d) {
            a.da[d] = da_of(reg0 + d);
            a.W[d] = w->W[l * D + d];
        }
        // layer 0 writes the caller's full-width dx directly
        a.site = nv; a.out = l == 0 ? dx : dxc_here; a.scatter = l == 0; a.D = D; a.B = B; a.G = G; a.ldo = kin;
        a.T = T; a.K = kin; a.tps = ((kin + 7) / 8 + 15) / 16; a.mtiles = P.mtiles;
        a.dense = !P.compact; a.s = P.s_nr[l];
        a.status = sync_status;
        a.big = std::is_same<E, bf16>::value && B >= 64 && use_gemm_big();
        launch_dx<E>(a, kin, st);
    };
    // weight and bias gradients (Eq. 11) of layer l: its problems join one
    // batch (row-sparse and full problems alike), one launch per batch
    WgBatch b;
    b.np = 0;
    b.status = sync_status;
    b.big = std::is_same<E, bf16>::value && wgrad_big_fits(B) && use_big() && (B >= 128 || big_mode() == 2) &&
            use_wgrad_big();
    auto add_wgrad = [&](const WgArgs& a) {
        if (b.np == WG_MAXP) {                 // full: launch it (its DA is complete)
            launch_wgrad<E>(b, st);
            b.np = 0;
        }
        b.p[b.np++] = a;
    };
    auto layer_wgrad = [&](int l, int reg0) {
        const int kin = P.kin(l);
        const SiteView nv = site_view(P, mbuf, P.site_nr(l));
        const void* XT = l == 0 ? (const void*)(R + P.r_xT) : (const void*)(R + P.rybufT(l - 1));
        for (int d = 0; d < D; ++d) {
            const int k = l * D + d;
            const char* rd = R + P.rdir(l, d);
            WgArgs a;
            memset(&a, 0, sizeof(a));
            a.actT = XT; a.tstride = (long)kin * BP; a.actT_first = nullptr; a.t_first = -1; a.shift = 0;
            a.daT = daT_of(reg0 + d);
            a.site = nv; a.K = kin; a.B = B; a.BP = BP; a.G = G; a.T = T;
            a.dense = !P.compact; a.s = P.s_nr[l];
            a.out = g->dW[k];
            a.db = g->db[k];                      // the bias gradient rides on the input-weight pass
            a.full = P.p_nr[l] == 0.0 || !P.compact;
            add_wgrad(a);

            WgArgs u = a;
            u.actT = rd + P.r_hrecT; u.tstride = (long)H * BP;
            u.actT_first = R + P.r_h0T + (size_t)k * H * BP * es;
            u.t_first = d == 0 ? 0 : T - 1;
            u.shift = d == 0 ? -1 : 1;
            u.site = site_view(P, mbuf, P.site_rh(l, d));
            u.K = H; u.s = P.s_rh[l];
            u.out = g->dU[k];
            u.db = nullptr;
            u.full = P.p_rh[l] == 0.0 || !P.compact;
            add_wgrad(u);
        }
    };
    auto flush_wgrad = [&]() {
        launch_wgrad<E>(b, st);
        b.np = 0;
    };

    // Unidirectional stack: every layer's BPTT in one persistent launch, with
    // a worker between layers l+1 and l forming dx of layer l+1 per step.
    const bool big_first = std::is_same<E, bf16>::value && big_mode() == 2;
    if (use_persistent() && use_stacked() && !big_first && D == 1 && L > 1 && 2 * L - 1 <= 8) {
        launch_bwd_init(nullptr, nullptr, nullptr, nullptr, 0, W + P.w_da, (int)es, G, P.mtiles, (long)L * T,
                        (long)P.das, sync_bar, sync_err, st);
        PBwdArgs pa;
        common_args(pa);
        pa.nslots = 2 * L - 1;
        for (int l = L - 1; l >= 0; --l) {
            const int slot = 2 * (L - 1 - l);             // layer l; its worker (dx of l for l-1) at slot + 1
            fill_layer(pa.d[slot], l, 0, l);
            if (l < L - 1) {
                pa.d[slot].above = slot - 1;
                pa.d[slot].dxw = (const float*)(W + P.w_dxw) + (size_t)l * T * B * H;
            }
            if (l > 0) {
                PBwdDir& wk = pa.d[slot + 1];
                wk.role = 1;
                wk.src = slot;
                wk.dir = 0;
                wk.above = -1;
                wk.Wup = w->W[l];
                wk.s_nr = P.s_nr[l];
                wk.nr_up = site_view(P, mbuf, P.site_nr(l));
                wk.dxw_out = (float*)(W + P.w_dxw) + (size_t)(l - 1) * T * B * H;
                wk.dh0 = dh0 + (size_t)l * B * H;         // unused by a worker (poisoning targets only)
                wk.dc0 = dc0 + (size_t)l * B * H;
            }
        }
        hipEvent_t e0 = nullptr, e1 = nullptr;
        const bool timed = timer_pair(KID_BWDP_, &e0, &e1);
        if (launch_bwd_persist<E>(pa, st, timed, e0, e1) == hipSuccess) {
            if (dx) layer_dx(0, 0, (float*)(W + P.w_dxc));
            for (int l = L - 1; l >= 0; --l) layer_wgrad(l, l);
            flush_wgrad();
            return hip_check("backward launch");
        }
        (void)hipGetLastError();              // does not fit: one layer at a time below
        if (timed) timer_unpair();
    }

    for (int l = L - 1; l >= 0; --l) {
        float* dhc = (float*)(W + P.w_dhc);
        float* dcs = (float*)(W + P.w_dc);
        launch_bwd_init(dhT ? dhT + (size_t)l * D * B * H : nullptr, dcT ? dcT + (size_t)l * D * B * H : nullptr,
                        dhc, dcs, (long)D * B * H, l == L - 1 ? (void*)(W + P.w_da) : nullptr, (int)es, G,
                        P.mtiles, (long)D * T, (long)P.das, sync_bar, sync_err, st);
        float* dxc_above = (float*)(W + P.w_dxc) + (size_t)((l + 1) & 1) * T * B * P.kin_max;
        float* dxc_here = (float*)(W + P.w_dxc) + (size_t)(l & 1) * T * B * P.kin_max;
        bool persistent_done = false;
        // the large-batch kernel, one launch per direction
        auto big = [&]() -> bool {
            if (!std::is_same<E, bf16>::value || !use_big()) return false;
            for (int d = 0; d < D; ++d) {
                PBwdArgs pa;
                common_args(pa);
                pa.nslots = 1;
                pa.lddx = l + 1 < L ? P.kin(l + 1) : 0;
                pa.part = (float*)(W + P.w_part);
                PBwdDir& pd = pa.d[0];
                fill_layer(pd, l, d, d);
                if (l < L - 1) {
                    pd.dxc = dxc_above;
                    pd.dxpos = site_view(P, mbuf, P.site_nr(l + 1)).pos + d * H;
                }
                hipEvent_t e0 = nullptr, e1 = nullptr;
                const bool timed = timer_pair(KID_BWDP_, &e0, &e1);
                if (launch_bwd_big(pa, st, timed, e0, e1) != hipSuccess) {
                    (void)hipGetLastError();
                    if (timed) timer_unpair();
                    return false;             // (the first direction: nothing was launched)
                }
            }
            return true;
        };
        if (use_persistent() && big_first) persistent_done = big();
        if (use_persistent() && !persistent_done) {
            PBwdArgs pa;
            common_args(pa);
            pa.nslots = D;
            pa.lddx = l + 1 < L ? P.kin(l + 1) : 0;
            for (int d = 0; d < D; ++d) {
                PBwdDir& pd = pa.d[d];
                fill_layer(pd, l, d, d);
                if (l < L - 1) {
                    pd.dxc = dxc_above;
                    pd.dxpos = site_view(P, mbuf, P.site_nr(l + 1)).pos + d * H;
                }
            }
            hipEvent_t e0 = nullptr, e1 = nullptr;
            const bool timed = timer_pair(KID_BWDP_, &e0, &e1);
            if (launch_bwd_persist<E>(pa, st, timed, e0, e1) == hipSuccess) {
                persistent_done = true;
            } else {
                (void)hipGetLastError();      // does not fit: the large-batch kernel, else per step
                if (timed) timer_unpair();
                persistent_done = big();
            }
        }
        // T pointwise steps plus one final pass (recurrent gradient of h0)
        for (int s = 0; s <= T && !persistent_done; ++s) {
            const bool final_pass = s == T;
            BwdArgs a;
            memset(&a, 0, sizeof(a));
            a.lengths = lengths; a.B = B; a.H = H; a.BP = BP; a.ldy = D * H;
            a.lddx = l + 1 < L ? P.kin(l + 1) : 0;
            a.tps = tps_h; a.has_next = s > 0; a.mtiles = P.mtiles; a.final_pass = final_pass; a.dense = !P.compact; a.s = P.s_rh[l];
            for (int d = 0; d < D; ++d) {
                const int k = l * D + d;
                const int t = final_pass ? -1 : (d == 0 ? T - 1 - s : s);   // BP order: reverse of FP
                const int tn = d == 0 ? T - s : s - 1;                        // step processed just before
                const int tp = d == 0 ? t - 1 : t + 1;                        // forward predecessor of t
                const char* rd = R + P.rdir(l, d);
                const SiteView rv = site_view(P, mbuf, P.site_rh(l, d));
                BwdDir& bd = a.d[d];
                bd.t = t;
                bd.U = w->U[k];
                bd.dhc = dhc + (size_t)d * B * H;
                bd.dcs = dcs + (size_t)d * B * H;
                if (s > 0) {
                    bd.da_next = (char*)da_of(d) + (size_t)tn * P.das * es;
                    bd.nmask = rv.mask + (size_t)tn * P.kmax;
                    bd.nkeep = rv.keep + (size_t)tn * P.kmax;
                    bd.ncount = rv.count + tn;
                    bd.ndrop = rv.drop + (size_t)tn * P.kmax;
                    bd.ndcount = rv.dcount + tn;
                    bd.nkseg = rv.kseg + (size_t)tn * 17;
                    bd.ndseg = rv.dseg + (size_t)tn * 17;
                }
                if (final_pass) {
                    bd.dh0 = dh0 + (size_t)k * B * H;
                    bd.dc0 = dc0 + (size_t)k * B * H;
                    continue;
                }
                bd.gates = (const float*)(rd + P.r_gates) + (size_t)t * B * G;
                bd.cres = (const float*)(rd + P.r_c) + (size_t)t * B * H;
                bd.cprev = s == T - 1 ? c0 + (size_t)k * B * H : (const float*)(rd + P.r_c) + (size_t)tp * B * H;
                if (l == L - 1) {
                    bd.dy = dy + (size_t)t * B * D * H + d * H;
                } else {
                    const SiteView sv = site_view(P, mbuf, P.site_nr(l + 1));
                    bd.dxc = dxc_above + (size_t)t * B * a.lddx;
                    bd.dxpos = sv.pos + (size_t)t * P.kmax + d * H;
                }
                bd.da = (char*)da_of(d) + (size_t)t * P.das * es;
                bd.daT = (char*)daT_of(d) + (size_t)t * G * BP * es;
            }
            launch_bwd<E>(a, D, st);
        }
        if (l > 0 || dx) layer_dx(l, 0, dxc_here);
        layer_wgrad(l, 0);
        flush_wgrad();                        // before the next layer reuses the DA regions
    }
    return hip_check("backward launch");
}

}  // namespace lsd

using namespace lsd;

// ---------------------------------------------------------------------------
// Output head (pre-FC output dropout, FC layer, softmax cross-entropy).
struct HeadPlan {
    int F, V, B, T, dtype, compact, sid, BP, mtiles;
    double p;
    float s;
    size_t esize, das;
    // mask buffer: one site, kmax = F
    size_t m_mask, m_keep, m_pos, m_count, m_drop, m_dcount, m_kseg, m_dseg, m_total;
    // workspace
    size_t w_yb, w_ybT, w_da, w_daT, w_lse, w_rowloss, w_rowok, w_ninv, w_total;
};

static int make_head_plan(const lstm_sd_head_dims* d, HeadPlan* p, const char** why) {
    if (!d) { *why = "head dims is NULL"; return LSTM_SD_EINVAL; }
    if (d->features < 1 || d->batch < 1 || d->seq_len < 1 || d->vocab < 1) {
        *why = "dimensions must be >= 1"; return LSTM_SD_EINVAL;
    }
    if (!(d->p_out >= 0.0 && d->p_out < 1.0)) { *why = "p_out must be in [0, 1)"; return LSTM_SD_EINVAL; }
    if (d->compact != 0 && d->compact != 1) { *why = "compact must be 0 or 1"; return LSTM_SD_EINVAL; }
    if (d->stream_id < 0) { *why = "stream_id must be >= 0"; return LSTM_SD_EINVAL; }
    if (d->dtype != LSTM_SD_DTYPE_F32 && d->dtype != LSTM_SD_DTYPE_BF16) {
        *why = "dtype must be 0 (f32) or 1 (bf16)"; return LSTM_SD_EUNSUPPORTED;
    }
    const size_t es = d->dtype == LSTM_SD_DTYPE_BF16 ? 2 : 4;
    if (d->features > LSTM_SD_MAX_K) { *why = "features must be <= LSTM_SD_MAX_K"; return LSTM_SD_EUNSUPPORTED; }
    if (d->vocab < 4 || d->vocab % 4) { *why = "vocab must be a multiple of 4"; return LSTM_SD_EUNSUPPORTED; }
    if ((size_t)d->features * d->vocab * es >= (1ull << 31)) {
        *why = "features*vocab*sizeof(dtype) must be < 2^31"; return LSTM_SD_EUNSUPPORTED;
    }
    if ((long)d->batch * d->seq_len > (1L << 24) || d->batch > 65536 || d->seq_len > 65535) {
        *why = "batch*seq_len too large"; return LSTM_SD_EUNSUPPORTED;
    }
    HeadPlan& q = *p;
    q.F = d->features; q.V = d->vocab; q.B = d->batch; q.T = d->seq_len; q.dtype = d->dtype;
    q.compact = d->compact; q.sid = d->stream_id; q.p = d->p_out; q.s = inv_keep(d->p_out);
    q.esize = es;
    q.BP = (q.B + 31) / 32 * 32;
    q.mtiles = (q.B + 15) / 16;
    q.das = (size_t)((q.V + 31) / 32) * q.mtiles * 512;
    const size_t A = 256, T = q.T, B = q.B, F = q.F, V = q.V, BP = q.BP;
    size_t off = 0;
    q.m_mask = off;   off = align_up(off + T * F, A);
    q.m_keep = off;   off = align_up(off + T * F * 4, A);
    q.m_pos = off;    off = align_up(off + T * F * 4, A);
    q.m_count = off;  off = align_up(off + T * 4, A);
    q.m_drop = off;   off = align_up(off + T * F * 4, A);
    q.m_dcount = off; off = align_up(off + T * 4, A);
    q.m_kseg = off;   off = align_up(off + T * 17 * 4, A);
    q.m_dseg = off;   off = align_up(off + T * 17 * 4, A);
    q.m_total = off;
    off = 0;
    q.w_yb = off;      off = align_up(off + T * B * F * es, A);
    q.w_ybT = off;     off = align_up(off + T * F * BP * es, A);
    q.w_da = off;      off = align_up(off + T * q.das * es, A);
    q.w_daT = off;     off = align_up(off + T * V * BP * es, A);
    q.w_lse = off;     off = align_up(off + T * B * 4, A);
    q.w_rowloss = off; off = align_up(off + T * B * 4, A);
    q.w_rowok = off;   off = align_up(off + T * B * 4, A);
    q.w_ninv = off;    off = align_up(off + 4, A);
    q.w_total = off;
    return LSTM_SD_OK;
}

static SiteView head_site(const HeadPlan& P, const void* mbuf) {
    const char* m = (const char*)mbuf;
    SiteView v;
    v.mask = (const uint8_t*)(m + P.m_mask);
    v.keep = (const int32_t*)(m + P.m_keep);
    v.pos = (const int32_t*)(m + P.m_pos);
    v.count = (const int32_t*)(m + P.m_count);
    v.drop = (const int32_t*)(m + P.m_drop);
    v.dcount = (const int32_t*)(m + P.m_dcount);
    v.kseg = (const int32_t*)(m + P.m_kseg);
    v.dseg = (const int32_t*)(m + P.m_dseg);
    v.kmax = P.F;
    return v;
}

template <typename E>
static void head_backward_impl(const HeadPlan& P, const void* W_fc, const int32_t* tgt, const int32_t* lengths,
                               const void* mbuf, const float* logits, float* loss, float* dy, float* dW, float* db,
                               char* W, hipStream_t st) {
    float* lse = (float*)(W + P.w_lse);
    float* ninv = (float*)(W + P.w_ninv);
    launch_ce_loss(logits, tgt, lengths, P.T, P.B, P.V, lse, (float*)(W + P.w_rowloss), (float*)(W + P.w_rowok), loss,
                   ninv, st);
    launch_ce_grad<E>(logits, tgt, lengths, lse, ninv, P.T, P.B, P.V, P.BP, P.mtiles, W + P.w_da, W + P.w_daT, st);
    const SiteView site = head_site(P, mbuf);
    DxArgs a;
    memset(&a, 0, sizeof(a));
    a.da[0] = W + P.w_da; a.W[0] = W_fc;
    a.site = site; a.out = dy; a.scatter = 1; a.D = 1; a.B = P.B; a.G = P.V; a.ldo = P.F;
    a.T = P.T; a.K = P.F; a.tps = ((P.F + 7) / 8 + 15) / 16; a.mtiles = P.mtiles;
    a.dense = !P.compact; a.s = P.s;
    launch_dx<E>(a, P.F, st);
    WgBatch b;
    memset(&b, 0, sizeof(b));
    b.np = 1;
    WgArgs& g = b.p[0];
    g.actT = W + P.w_ybT; g.tstride = (long)P.F * P.BP; g.actT_first = nullptr; g.t_first = -1; g.shift = 0;
    g.daT = W + P.w_daT;
    g.site = site; g.K = P.F; g.B = P.B; g.BP = P.BP; g.G = P.V; g.T = P.T;
    g.dense = !P.compact; g.s = P.s;
    g.out = dW; g.db = db;
    g.full = P.p == 0.0 || !P.compact;
    launch_wgrad<E>(b, st);
}

extern "C" {

int lstm_sd_version(void) { return 1; }

const char* lstm_sd_last_error(void) { return g_err.c_str(); }

size_t lstm_sd_mask_bytes(const lstm_sd_dims* dims) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) { fail(rc, why); return 0; }
    return P.m_total;
}

size_t lstm_sd_reserve_bytes(const lstm_sd_dims* dims) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) { fail(rc, why); return 0; }
    return P.r_total;
}

size_t lstm_sd_workspace_bytes(const lstm_sd_dims* dims) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) { fail(rc, why); return 0; }
    return P.w_total;
}

int lstm_sd_mask_layout_get(const lstm_sd_dims* dims, lstm_sd_mask_layout* out) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!out) return fail(LSTM_SD_EINVAL, "out is NULL");
    out->sites = P.sites; out->kmax = P.kmax; out->seq_len = P.T; out->reserved = 0;
    out->mask_off = P.m_mask; out->keep_off = P.m_keep; out->pos_off = P.m_pos;
    out->count_off = P.m_count; out->drop_off = P.m_drop; out->dcount_off = P.m_dcount;
    out->kseg_off = P.m_kseg; out->dseg_off = P.m_dseg;
    out->total_bytes = P.m_total;
    return LSTM_SD_OK;
}

int lstm_sd_mask_generate(const lstm_sd_dims* dims, uint64_t seed, uint64_t step, void* mask_buf,
                          size_t mask_bytes, void* stream) {
    return do_masks(dims, seed, step, mask_buf, mask_bytes, stream, 1);
}

int lstm_sd_mask_generate_fixed(const lstm_sd_dims* dims, uint64_t seed, uint64_t step, void* mask_buf,
                                size_t mask_bytes, void* stream) {
    return do_masks(dims, seed, step, mask_buf, mask_bytes, stream, 1, 1);
}

int lstm_sd_mask_compact(const lstm_sd_dims* dims, void* mask_buf, size_t mask_bytes, void* stream) {
    return do_masks(dims, 0, 0, mask_buf, mask_bytes, stream, 0);
}

int lstm_sd_forward(const lstm_sd_dims* dims, const lstm_sd_weights* w, const void* x, const int32_t* lengths,
                    const void* h0, const float* c0, const void* mask_buf, size_t mask_bytes, float* y,
                    float* hT, float* cT, void* reserve, size_t reserve_bytes, void* workspace,
                    size_t workspace_bytes, void* stream) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!w || !w->W || !w->U || !w->b) return fail(LSTM_SD_EINVAL, "weights is NULL");
    for (int k = 0; k < P.L * P.D; ++k)
        if (!w->W[k] || !w->U[k] || !w->b[k]) return fail(LSTM_SD_EINVAL, "a weight pointer is NULL");
    if (!x || !h0 || !c0 || !mask_buf || !y || !hT || !cT || !reserve || !workspace)
        return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_mask_bytes()");
    if (reserve_bytes < P.r_total) return fail(LSTM_SD_EWORKSPACE, "reserve_bytes smaller than lstm_sd_reserve_bytes()");
    if (workspace_bytes < P.w_total) return fail(LSTM_SD_EWORKSPACE, "workspace_bytes smaller than lstm_sd_workspace_bytes()");
    if (setup_kernel_attributes()) return fail(LSTM_SD_EHIP, "hipFuncSetAttribute failed");
    hipStream_t st = (hipStream_t)stream;
    if (P.dtype == LSTM_SD_DTYPE_BF16)
        return forward_impl<bf16>(P, w, x, lengths, h0, c0, mask_buf, y, hT, cT, reserve, workspace, st);
    return forward_impl<float>(P, w, x, lengths, h0, c0, mask_buf, y, hT, cT, reserve, workspace, st);
}

int lstm_sd_backward(const lstm_sd_dims* dims, const lstm_sd_weights* w, const void* x, const int32_t* lengths,
                     const void* h0, const float* c0, const void* mask_buf, size_t mask_bytes,
                     const void* reserve, size_t reserve_bytes, const float* dy, const float* dhT,
                     const float* dcT, float* dx, float* dh0, float* dc0, const lstm_sd_grads* g,
                     void* workspace, size_t workspace_bytes, void* stream) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!w || !w->W || !w->U || !w->b) return fail(LSTM_SD_EINVAL, "weights is NULL");
    if (!g || !g->dW || !g->dU || !g->db) return fail(LSTM_SD_EINVAL, "grads is NULL");
    for (int k = 0; k < P.L * P.D; ++k) {
        if (!w->W[k] || !w->U[k] || !w->b[k]) return fail(LSTM_SD_EINVAL, "a weight pointer is NULL");
        if (!g->dW[k] || !g->dU[k] || !g->db[k]) return fail(LSTM_SD_EINVAL, "a gradient pointer is NULL");
    }
    if (!x || !h0 || !c0 || !mask_buf || !reserve || !dy || !dh0 || !dc0 || !workspace)
        return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_mask_bytes()");
    if (reserve_bytes < P.r_total) return fail(LSTM_SD_EWORKSPACE, "reserve_bytes smaller than lstm_sd_reserve_bytes()");
    if (workspace_bytes < P.w_total) return fail(LSTM_SD_EWORKSPACE, "workspace_bytes smaller than lstm_sd_workspace_bytes()");
    if (setup_kernel_attributes()) return fail(LSTM_SD_EHIP, "hipFuncSetAttribute failed");
    hipStream_t st = (hipStream_t)stream;
    if (P.dtype == LSTM_SD_DTYPE_BF16)
        return backward_impl<bf16>(P, w, lengths, c0, mask_buf, reserve, dy, dhT, dcT, dx, dh0, dc0, g,
                                   workspace, st);
    return backward_impl<float>(P, w, lengths, c0, mask_buf, reserve, dy, dhT, dcT, dx, dh0, dc0, g,
                                workspace, st);
}

int lstm_sd_mse_grad(const lstm_sd_dims* dims, const float* y, const float* target, const int32_t* lengths,
                     float* dy, float* loss, void* workspace, size_t workspace_bytes, void* stream) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!y || !target || !dy || !loss || !workspace) return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (workspace_bytes < P.w_total) return fail(LSTM_SD_EWORKSPACE, "workspace_bytes smaller than lstm_sd_workspace_bytes()");
    float* partial = (float*)((char*)workspace + P.w_loss);
    launch_mse(y, target, lengths, dy, partial, 1024, loss, P.T, P.B, P.D * P.H, (hipStream_t)stream);
    return hip_check("mse launch");
}

int lstm_sd_embedding_backward(const lstm_sd_dims* dims, const int32_t* tokens, int vocab, const float* dx,
                               const void* mask_buf, size_t mask_bytes, float* d_emb, void* stream) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!tokens || !dx || !mask_buf || !d_emb) return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (vocab <= 0) return fail(LSTM_SD_EINVAL, "vocab must be positive");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_mask_bytes()");
    const SiteView nr0 = site_view(P, mask_buf, P.site_nr(0));
    launch_emb_grad(tokens, P.T * P.B, P.B, vocab, dx, nr0, P.I, d_emb, (hipStream_t)stream);
    return hip_check("embedding gradient launch");
}

size_t lstm_sd_head_mask_bytes(const lstm_sd_head_dims* hd) {
    HeadPlan P; const char* why = nullptr;
    if (int rc = make_head_plan(hd, &P, &why)) { fail(rc, why); return 0; }
    return P.m_total;
}

size_t lstm_sd_head_workspace_bytes(const lstm_sd_head_dims* hd) {
    HeadPlan P; const char* why = nullptr;
    if (int rc = make_head_plan(hd, &P, &why)) { fail(rc, why); return 0; }
    return P.w_total;
}

int lstm_sd_head_mask_layout_get(const lstm_sd_head_dims* hd, lstm_sd_mask_layout* out) {
    HeadPlan P; const char* why = nullptr;
    if (int rc = make_head_plan(hd, &P, &why)) return fail(rc, why);
    if (!out) return fail(LSTM_SD_EINVAL, "out is NULL");
    out->sites = 1; out->kmax = P.F; out->seq_len = P.T; out->reserved = 0;
    out->mask_off = P.m_mask; out->keep_off = P.m_keep; out->pos_off = P.m_pos;
    out->count_off = P.m_count; out->drop_off = P.m_drop; out->dcount_off = P.m_dcount;
    out->kseg_off = P.m_kseg; out->dseg_off = P.m_dseg;
    out->total_bytes = P.m_total;
    return LSTM_SD_OK;
}

int lstm_sd_head_mask_generate(const lstm_sd_head_dims* hd, uint64_t seed, uint64_t step, void* mask_buf,
                               size_t mask_bytes, void* stream) {
    HeadPlan P; const char* why = nullptr;
    if (int rc = make_head_plan(hd, &P, &why)) return fail(rc, why);
    if (!mask_buf) return fail(LSTM_SD_EINVAL, "mask_buf is NULL");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_head_mask_bytes()");
    MaskArgs a;
    memset(&a, 0, sizeof(a));
    char* m = (char*)mask_buf;
    a.mask = (uint8_t*)(m + P.m_mask);
    a.keep = (int32_t*)(m + P.m_keep);
    a.pos = (int32_t*)(m + P.m_pos);
    a.count = (int32_t*)(m + P.m_count);
    a.drop = (int32_t*)(m + P.m_drop);
    a.dcount = (int32_t*)(m + P.m_dcount);
    a.kseg = (int32_t*)(m + P.m_kseg);
    a.dseg = (int32_t*)(m + P.m_dseg);
    a.T = P.T; a.kmax = P.F; a.compact = P.compact; a.generate = 1;
    a.seed = seed; a.step = step;
    a.K[0] = P.F;
    a.sid[0] = P.sid;
    a.thr[0] = threshold64(P.p);
    launch_mask_build(a, 1, (hipStream_t)stream);
    return hip_check("head mask kernel launch");
}

int lstm_sd_head_forward(const lstm_sd_head_dims* hd, const void* W_fc, const float* b_fc, const float* y,
                         const void* mask_buf, size_t mask_bytes, float* logits, void* workspace,
                         size_t workspace_bytes, void* stream) {
    HeadPlan P; const char* why = nullptr;
    if (int rc = make_head_plan(hd, &P, &why)) return fail(rc, why);
    if (!W_fc || !b_fc || !y || !mask_buf || !logits || !workspace)
        return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_head_mask_bytes()");
    if (workspace_bytes < P.w_total)
        return fail(LSTM_SD_EWORKSPACE, "workspace_bytes smaller than lstm_sd_head_workspace_bytes()");
    hipStream_t st = (hipStream_t)stream;
    char* W = (char*)workspace;
    FxArgs f;
    memset(&f, 0, sizeof(f));
    f.X = W + P.w_yb; f.ldx = P.F; f.W = W_fc; f.K = P.F; f.bias = b_fc; f.site = head_site(P, mask_buf);
    f.Gx = logits; f.B = P.B; f.G = P.V; f.T = P.T; f.dense = !P.compact; f.s = P.s;
    if (P.dtype == LSTM_SD_DTYPE_BF16) {
        launch_head_prep<bf16>(y, W + P.w_yb, W + P.w_ybT, P.T, P.B, P.F, P.BP, st);
        launch_fx<bf16>(f, st);
    } else {
        launch_head_prep<float>(y, W + P.w_yb, W + P.w_ybT, P.T, P.B, P.F, P.BP, st);
        launch_fx<float>(f, st);
    }
    return hip_check("head forward launch");
}

int lstm_sd_head_backward(const lstm_sd_head_dims* hd, const void* W_fc, const int32_t* targets,
                          const int32_t* lengths, const void* mask_buf, size_t mask_bytes, const float* logits,
                          float* loss, float* dy, float* dW_fc, float* db_fc, void* workspace,
                          size_t workspace_bytes, void* stream) {
    HeadPlan P; const char* why = nullptr;
    if (int rc = make_head_plan(hd, &P, &why)) return fail(rc, why);
    if (!W_fc || !targets || !mask_buf || !logits || !loss || !dy || !dW_fc || !db_fc || !workspace)
        return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_head_mask_bytes()");
    if (workspace_bytes < P.w_total)
        return fail(LSTM_SD_EWORKSPACE, "workspace_bytes smaller than lstm_sd_head_workspace_bytes()");
    if (setup_kernel_attributes()) return fail(LSTM_SD_EHIP, "hipFuncSetAttribute failed");
    hipStream_t st = (hipStream_t)stream;
    if (P.dtype == LSTM_SD_DTYPE_BF16)
        head_backward_impl<bf16>(P, W_fc, targets, lengths, mask_buf, logits, loss, dy, dW_fc, db_fc,
                                 (char*)workspace, st);
    else
        head_backward_impl<float>(P, W_fc, targets, lengths, mask_buf, logits, loss, dy, dW_fc, db_fc,
                                  (char*)workspace, st);
    return hip_check("head backward launch");
}

static const char* case1_check(int T, int B, int K, double p) {
    if (T < 1 || B < 1 || K < 1) return "dimensions must be >= 1";
    if (!(p >= 0.0 && p < 1.0)) return "p must be in [0, 1)";
    if ((long)T * B > (1L << 24) || B > 65536 || T > 65535) return "seq_len*batch too large";
    return nullptr;
}

int lstm_sd_case1_dropout(int32_t seq_len, int32_t batch, int32_t features, int32_t src_dtype, const void* src,
                          int32_t dst_dtype, void* dst, uint8_t* mask, uint64_t seed, uint64_t step, int32_t stream_id,
                          double p, void* stream) {
    if (const char* why = case1_check(seq_len, batch, features, p)) return fail(LSTM_SD_EINVAL, why);
    if (stream_id < 0) return fail(LSTM_SD_EINVAL, "stream_id must be >= 0");
    if ((src_dtype != LSTM_SD_DTYPE_F32 && src_dtype != LSTM_SD_DTYPE_BF16) ||
        (dst_dtype != LSTM_SD_DTYPE_F32 && dst_dtype != LSTM_SD_DTYPE_BF16))
        return fail(LSTM_SD_EUNSUPPORTED, "dtypes must be 0 (f32) or 1 (bf16)");
    if (!src || !dst || !mask) return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    launch_case1_drop(src_dtype == LSTM_SD_DTYPE_F32, dst_dtype == LSTM_SD_DTYPE_BF16, src, dst, mask, seq_len, batch,
                      features, seed, step, (uint64_t)stream_id, threshold64(p), inv_keep(p), (hipStream_t)stream);
    return hip_check("case-I dropout launch");
}

int lstm_sd_case1_dropout_backward(int32_t seq_len, int32_t batch, int32_t features, const float* dx,
                                   const uint8_t* mask, double p, float* dsrc, void* stream) {
    if (const char* why = case1_check(seq_len, batch, features, p)) return fail(LSTM_SD_EINVAL, why);
    if (!dx || !mask || !dsrc) return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    launch_case1_undrop(dx, mask, dsrc, (long)seq_len * batch * features, inv_keep(p), (hipStream_t)stream);
    return hip_check("case-I dropout backward launch");
}

// ---------------------------------------------------------------------------
// The forward pass with the library's own workspace, for callers that cannot
// allocate.  `scratch` is a file-scope device array: each GPU the library
// runs on holds its own copy until the process ends.  In host code its name
// is not a device address; the address of the current device's copy comes
// from hipGetSymbolAddress, taken once per device on the first call there,
// and only that pointer reaches kernels.
static __device__ __align__(256) char scratch[LSTM_SD_STATIC_WORKSPACE_MAX];

static int scratch_ptr(void** out) {
    constexpr int MAXDEV = 64;
    static std::mutex mu;
    static void* ptr[MAXDEV] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(LSTM_SD_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    if (dev < 0 || dev >= MAXDEV) return fail(LSTM_SD_EUNSUPPORTED, "device index beyond the static workspace table");
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(LSTM_SD_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        ptr[dev] = p;
    }
    *out = ptr[dev];
    return LSTM_SD_OK;
}

int lstm_sd_forward_static(const lstm_sd_dims* dims, const lstm_sd_weights* w, const void* x, const int32_t* lengths,
                           const void* h0, const float* c0, const void* mask_buf, size_t mask_bytes, float* y,
                           float* hT, float* cT, void* reserve, size_t reserve_bytes, void* stream) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (P.w_total > LSTM_SD_STATIC_WORKSPACE_MAX)
        return fail(LSTM_SD_EUNSUPPORTED, "lstm_sd_workspace_bytes(dims) exceeds LSTM_SD_STATIC_WORKSPACE_MAX");
    if (!w || !w->W || !w->U || !w->b) return fail(LSTM_SD_EINVAL, "weights is NULL");
    for (int k = 0; k < P.L * P.D; ++k)
        if (!w->W[k] || !w->U[k] || !w->b[k]) return fail(LSTM_SD_EINVAL, "a weight pointer is NULL");
    if (!x || !h0 || !c0 || !mask_buf || !y || !hT || !cT || !reserve)
        return fail(LSTM_SD_EINVAL, "a required pointer is NULL");
    if (mask_bytes < P.m_total) return fail(LSTM_SD_EWORKSPACE, "mask_bytes smaller than lstm_sd_mask_bytes()");
    if (reserve_bytes < P.r_total) return fail(LSTM_SD_EWORKSPACE, "reserve_bytes smaller than lstm_sd_reserve_bytes()");
    void* ws = nullptr;
    if ((rc = scratch_ptr(&ws))) return rc;
    if (setup_kernel_attributes()) return fail(LSTM_SD_EHIP, "hipFuncSetAttribute failed");
    hipStream_t st = (hipStream_t)stream;
    if (P.dtype == LSTM_SD_DTYPE_BF16)
        return forward_impl<bf16>(P, w, x, lengths, h0, c0, mask_buf, y, hT, cT, reserve, ws, st);
    return forward_impl<float>(P, w, x, lengths, h0, c0, mask_buf, y, hT, cT, reserve, ws, st);
}

int lstm_sd_status(const lstm_sd_dims* dims, const void* workspace, size_t workspace_bytes, void* stream) {
    Plan P; const char* why = nullptr;
    int rc = make_plan(dims, &P, &why);
    if (rc) return fail(rc, why);
    if (!workspace) return fail(LSTM_SD_EINVAL, "workspace is NULL");
    if (workspace_bytes < P.w_total) return fail(LSTM_SD_EWORKSPACE, "workspace_bytes smaller than lstm_sd_workspace_bytes()");
    int v = 0;
    hipError_t e = hipStreamSynchronize((hipStream_t)stream);
    if (e == hipSuccess) e = hipMemcpy(&v, (const char*)workspace + P.w_sync + SYNC_STATUS_OFS, sizeof(v), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(LSTM_SD_EHIP, std::string("status read: ") + hipGetErrorString(e));
    if (v == 0) return LSTM_SD_OK;
    std::string m = "grid barrier time-out in the";
    if (v & STATUS_FWD) m += " forward";
    if ((v & STATUS_FWD) && (v & STATUS_BWD)) m += " and the";
    if (v & STATUS_BWD) m += " backward";
    m += " pass of the last step: its outputs were written as NaN";
    return fail(LSTM_SD_EHIP, m);
}

int lstm_sd_set_barrier_timeout(double seconds) {
    if (!(seconds == seconds)) return fail(LSTM_SD_EINVAL, "time-out is NaN");
    g_timeout_s.store(seconds < 0.0 ? -1.0 : seconds);
    return LSTM_SD_OK;
}

int lstm_sd_kernel_timer_start(const char* kernel) {
    if (kernel_timer_start(kernel)) return fail(LSTM_SD_EINVAL, std::string("unknown kernel name: ") + (kernel ? kernel : "(null)"));
    return LSTM_SD_OK;
}

int lstm_sd_kernel_timer_stop(double* total_ms, int64_t* launches) {
    if (kernel_timer_stop(total_ms, launches)) return fail(LSTM_SD_EHIP, "kernel timer: HIP event error");
    return LSTM_SD_OK;
}

}  // extern "C"
