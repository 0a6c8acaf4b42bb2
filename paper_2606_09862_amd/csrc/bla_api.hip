// Host side of the C ABI declared in include/bla.h: argument validation, the
// launch plan (segments, summarised blocks, workspace layout) and the launches.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>

#include <hip/hip_runtime.h>

#include "bla.h"
#include "bla_plan.h"

namespace {

using namespace bla;

constexpr size_t kAlign = 256;
constexpr size_t kMaxSummaryBytes = size_t(256) << 20;  // cap on per-block summary scratch
constexpr int kMaxPairSegments = 16;                     // segments per sequence on the pair kernel

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int pad_modes(int M) { return M <= 16 ? 16 : M <= 32 ? 32 : M <= 64 ? 64 : M <= 128 ? 128 : -1; }
int pad_slots(int S) { return S <= 32 ? 32 : S <= 64 ? 64 : S <= 128 ? 128 : S <= 256 ? 256 : -1; }

// Compute units of the current device, cached per device.  Concurrent first calls may both
// query the runtime; they store the same value, and the atomic makes that race benign.
int device_cu_count()
{
    static std::atomic<int> cache[128];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 128) return 256;
    int n = cache[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        cache[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Record of the tables last built into each workspace: (device, workspace address) -> key of
// the tables' contents.  A call with reuse_tables = 1 skips the table kernel when the record
// of its workspace matches its key.  A fixed ring of records; the oldest is overwritten.
struct TableRecord {
    int dev;
    const void* ws;
    uint64_t key;
};
constexpr int kTableRecords = 64;
std::mutex g_table_mu;
TableRecord g_table_rec[kTableRecords];
int g_table_next = 0;

uint64_t fnv_mix(uint64_t h, const void* data, size_t n)
{
    const unsigned char* c = (const unsigned char*)data;
    for (size_t i = 0; i < n; ++i) h = (h ^ c[i]) * 1099511628211ull;
    return h;
}

bool tables_recorded(int dev, const void* ws, uint64_t key)
{
    std::lock_guard<std::mutex> lk(g_table_mu);
    for (int i = 0; i < kTableRecords; ++i)
        if (g_table_rec[i].ws == ws && g_table_rec[i].dev == dev) return g_table_rec[i].key == key;
    return false;
}

void tables_record(int dev, const void* ws, uint64_t key)
{
    std::lock_guard<std::mutex> lk(g_table_mu);
    for (int i = 0; i < kTableRecords; ++i)
        if (g_table_rec[i].ws == ws && g_table_rec[i].dev == dev) {
            g_table_rec[i].key = key;
            return;
        }
    g_table_rec[g_table_next] = TableRecord{dev, ws, key};
    g_table_next = (g_table_next + 1) % kTableRecords;
}

bool aligned16(const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; }

// Shape checks shared by every entry point (no pointers).
bla_status check_shape(const bla_params* p, bool step)
{
    if (!p) return BLA_ERR_INVALID_ARG;
    if (p->B < 0 || p->H < 0 || (!step && p->L < 0)) return BLA_ERR_INVALID_ARG;
    if (p->d_k <= 0 || p->d_v <= 0 || p->M <= 0 || p->S <= 0 || p->t0 < 0) return BLA_ERR_INVALID_ARG;
    if (p->io_dtype != BLA_F32 && p->io_dtype != BLA_BF16) return BLA_ERR_INVALID_ARG;
    if (!isfinite(p->scale)) return BLA_ERR_INVALID_ARG;
    if (p->phase_anchor != 0 && p->phase_anchor != 1) return BLA_ERR_INVALID_ARG;
    if (p->reuse_tables != 0 && p->reuse_tables != 1) return BLA_ERR_INVALID_ARG;
    if (p->chunk != 0 && p->chunk != 16 && p->chunk != 32 && p->chunk != 64 && p->chunk != 128)
        return BLA_ERR_UNSUPPORTED;
    if (p->d_k != p->d_v) return BLA_ERR_UNSUPPORTED;
    if (p->d_k != 32 && p->d_k != 64 && p->d_k != 128) return BLA_ERR_UNSUPPORTED;
    const int MP = pad_modes(p->M), SP = pad_slots(p->S);
    if (MP < 0 || SP < 0) return BLA_ERR_UNSUPPORTED;
    if (SP > (2 * MP > 32 ? 2 * MP : 32)) return BLA_ERR_UNSUPPORTED;
    if (!step && !forward_supported(p->io_dtype == BLA_BF16, p->d_k, MP, SP, p->chunk ? p->chunk : kChunk))
        return BLA_ERR_UNSUPPORTED;
    if ((long long)p->B * p->H > (1ll << 31) / 4) return BLA_ERR_UNSUPPORTED;
    return BLA_OK;
}

bla_status check_periods(const bla_params* p, const double* T)
{
    if (p->H > 0 && !T) return BLA_ERR_INVALID_ARG;
    for (int h = 0; h < p->H; ++h)
        if (!isfinite(T[h]) || T[h] <= 0.0 || T[h] > 1e9) return BLA_ERR_INVALID_ARG;
    return BLA_OK;
}

void make_plan(const bla_params* p, bool step, Plan* pl)
{
    memset(pl, 0, sizeof(*pl));
    pl->B = p->B;
    pl->H = p->H;
    pl->L = step ? 1 : p->L;
    pl->D = p->d_k;
    pl->M = p->M;
    pl->S = p->S;
    pl->MP = pad_modes(p->M);
    pl->SP = pad_slots(p->S);
    // a decode step does not depend on the chunk length; its tables use the default's layout
    pl->C = step || p->chunk == 0 ? kChunk : p->chunk;
    pl->bf16 = p->io_dtype == BLA_BF16;
    pl->t0 = p->t0;
    pl->anchor = p->phase_anchor;
    pl->scale = p->scale != 0.f ? p->scale : 1.f / sqrtf((float)p->d_k);
    pl->unit_floats = (size_t)4 * pl->MP * pl->D;
    const long long units = (long long)p->B * p->H;
    pl->nch = step ? 1 : (p->L + pl->C - 1) / pl->C;
    pl->nseg = 1;
    pl->cps = pl->nch;
    pl->cpb = pl->nch;
    pl->nbs = 0;
    pl->upw = 1;
    pl->pair = 0;
    if (!step && pl->C == kChunk) {  // the pair kernels run 64-token chunks only
        const int pu = forward_units_per_wg(pl->bf16, pl->D, pl->MP, pl->SP);
        pl->upw = pu > 0 ? pu : 1;
        pl->pair = pu > 0;
    }
    if (!step && units > 0 && pl->nch > 1) {
        const int cus = device_cu_count();
        // The pair kernel combines every preceding segment summary in each unit's prologue,
        // which reads O(nseg^2) summaries per sequence.  Where filling the device would take
        // more than kMaxPairSegments segments (few, long sequences), the one-unit kernels run
        // instead: per-block summaries and a scan, linear in the number of segments.
        if (pl->pair && units * kMaxPairSegments < (long long)cus * pl->upw) {
            pl->pair = 0;
            pl->upw = 1;
        }
        const long long target = (long long)cus * pl->upw;  // units that fill every CU once
        if (units < target) {
            long long want = (target + units - 1) / units;
            int nseg = (int)(want < pl->nch ? want : pl->nch);
            int cps = (pl->nch + nseg - 1) / nseg;
            nseg = (pl->nch + cps - 1) / cps;
            pl->nseg = nseg;
            pl->cps = cps;
            if (nseg > 1) {
                // Blocks per segment: enough summary workgroups to fill the device, within
                // the scratch cap; always a divisor of cps.
                // The pair kernel combines the summaries itself: one block per segment.
                // bf16 64-token summaries run D/32 column-slice workgroups per block.
                int bps = 1;
                const size_t unit_bytes = pl->unit_floats * sizeof(float);
                const long long slices = pl->bf16 && pl->C == kChunk ? pl->D / 32 : 1;
                while (!pl->pair && units * (nseg - 1) * bps * slices < 2 * cus && cps % (2 * bps) == 0 &&
                       (size_t)units * (nseg - 1) * (2 * bps) * unit_bytes <= kMaxSummaryBytes)
                    bps *= 2;
                pl->cpb = cps / bps;
                pl->nbs = (nseg - 1) * bps;
            }
        }
    }
    const size_t esz = pl->bf16 ? 2 : 4;
    const size_t H = (size_t)p->H, C = (size_t)pl->C, MP2 = 2 * (size_t)pl->MP, SP = (size_t)pl->SP;
    size_t off = 0;
    pl->off_E32 = off;    off = align_up(off + H * (C + 1) * MP2 * 4);
    pl->off_EbarT = off;  off = align_up(off + H * MP2 * C * esz);
    pl->off_ErevT = off;  off = align_up(off + H * MP2 * C * esz);
    pl->off_Etab = off;   off = align_up(off + H * C * MP2 * esz);
    pl->off_ABs = off;    off = align_up(off + SP * MP2 * esz);
    pl->off_ABm = off;    off = align_up(off + MP2 * SP * esz);
    pl->off_theta = off;  off = align_up(off + H * SP * 4);
    pl->off_rotblk = off; off = align_up(off + H * MP2 * 4);
    pl->off_trig = off;   off = align_up(off + 2 * SP * 4);
    pl->off_rperiod = off; off = align_up(off + H * 8);
    pl->off_period = off; off = align_up(off + H * 8);
    pl->off_summ = off;   off = align_up(off + (size_t)units * pl->nbs * pl->unit_floats * 4);
    const size_t ncarry = pl->pair ? 0 : (size_t)(pl->nseg - 1);  // the pair kernel needs no carries
    pl->off_carry = off;  off = align_up(off + (size_t)units * ncarry * pl->unit_floats * 4);
    // the bf16 d = M = 128 forward kernel with 64 or 128 slots reads its tables as fragments
    pl->fragtab = !step && pl->bf16 && !pl->pair && pl->C == kChunk && pl->D == 128 && pl->MP == 128 &&
                  (pl->SP == 64 || pl->SP == 128);
    const size_t fab = pl->fragtab ? SP * MP2 * esz : 0, fh = pl->fragtab ? H * C * MP2 * esz : 0;
    pl->off_fABs = off;   off = align_up(off + fab);
    pl->off_fABm = off;   off = align_up(off + fab);
    pl->off_fEtab = off;  off = align_up(off + fh);
    pl->off_fEbar = off;  off = align_up(off + fh);
    pl->off_fErev = off;  off = align_up(off + fh);
    pl->off_fTw = off;    off = align_up(off + fh);
    pl->total = off;
}

// step: a decode step needs the phase rows j = 0, 1 only.  reuse: skip the launch when the
// library's record says this workspace already holds exactly these tables.
bla_status build_tables(const Plan& pl, const double* T, char* ws, hipStream_t s, bool step, int reuse)
{
    // key: everything the tables' contents and layout depend on
    int32_t f[14] = {pl.H, pl.M, pl.S, pl.MP, pl.SP, pl.C, pl.bf16, pl.anchor, pl.pair, step ? 2 : pl.C + 1,
                     pl.cpb * pl.C, 0, step ? 0 : pl.fragtab, 0};
    const float tab_scale = pl.pair ? 1.f : pl.scale;
    memcpy(&f[11], &tab_scale, sizeof(float));
    uint64_t key = fnv_mix(1469598103934665603ull, f, sizeof(f));
    for (int h = 0; h < pl.H; ++h) {
        const double tmin = 2.0 * pl.M - 1.0, Tc = T[h] < tmin ? tmin : T[h];
        key = fnv_mix(key, &Tc, sizeof(Tc));
    }
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return BLA_ERR_HIP;
    if (reuse && tables_recorded(dev, ws, key)) return BLA_OK;
    for (int h0 = 0; h0 < pl.H; h0 += kMaxHeadsPerTableLaunch) {
        TableArgs a;
        memset(&a, 0, sizeof(a));
        a.E32 = (float*)(ws + pl.off_E32);
        a.EbarT = ws + pl.off_EbarT;
        a.ErevT = ws + pl.off_ErevT;
        a.Etab = ws + pl.off_Etab;
        a.ABs = ws + pl.off_ABs;
        a.ABm = ws + pl.off_ABm;
        a.theta = (int*)(ws + pl.off_theta);
        a.rotblk = (float*)(ws + pl.off_rotblk);
        a.M = pl.M;
        a.S = pl.S;
        a.MP = pl.MP;
        a.SP = pl.SP;
        a.C = pl.C;
        a.Lblk = pl.cpb * pl.C;
        a.h0 = h0;
        a.nh = pl.H - h0 < kMaxHeadsPerTableLaunch ? pl.H - h0 : kMaxHeadsPerTableLaunch;
        a.with_shared = h0 == 0;
        a.conj_tab = pl.pair;
        a.jrows = step ? 2 : pl.C + 1;
        a.trig = (float*)(ws + pl.off_trig);
        a.rperiod = (double*)(ws + pl.off_rperiod);
        a.period = (double*)(ws + pl.off_period);
        a.negB = pl.anchor;
        a.scale = pl.pair ? 1.f : pl.scale;  // the pair kernel reads A | B unscaled
        for (int i = 0; i < a.nh; ++i) {
            const double tmin = 2.0 * pl.M - 1.0;
            a.T[i] = T[h0 + i] < tmin ? tmin : T[h0 + i];  // clamp, as Alg. 1 and Alg. 3 do
        }
        if (launch_tables(a, pl.bf16, s) != hipSuccess) return BLA_ERR_HIP;
    }
    if (!step && pl.fragtab) {
        FragTabArgs fa;
        fa.ABs = ws + pl.off_ABs;
        fa.ABm = ws + pl.off_ABm;
        fa.Etab = ws + pl.off_Etab;
        fa.EbarT = ws + pl.off_EbarT;
        fa.ErevT = ws + pl.off_ErevT;
        fa.fABs = ws + pl.off_fABs;
        fa.fABm = ws + pl.off_fABm;
        fa.fEtab = ws + pl.off_fEtab;
        fa.fEbar = ws + pl.off_fEbar;
        fa.fErev = ws + pl.off_fErev;
        fa.fTw = ws + pl.off_fTw;
        fa.H = pl.H;
        fa.C = pl.C;
        fa.MP = pl.MP;
        fa.SP = pl.SP;
        if (launch_fragtab(fa, s) != hipSuccess) return BLA_ERR_HIP;
    }
    tables_record(dev, ws, key);
    return BLA_OK;
}

// Decay form: the tables of a decode-step plan plus the segment summaries.  Sequences are
// cut into segments (a multiple of 16 tokens, at least 32) until the forward launch has
// about two waves per SIMD, within a 512 MB cap on the summaries.
struct DecayPlan {
    Plan pl;
    int nseg, seg_len;
    size_t off_summ, off_gmap, off_glen, off_gE, off_gB, total;
};

void make_decay_plan(const bla_params* p, DecayPlan* dp)
{
    make_plan(p, true, &dp->pl);
    const int L = p->L > 0 ? p->L : 0;
    const long long units = (long long)p->B * p->H;
    const int SP = dp->pl.SP, D = dp->pl.D;
    const size_t sf_bytes = ((size_t)2 * SP * D + SP) * sizeof(float);
    int nseg = 1, seg_len = L > 0 ? L : 1;
    if (units > 0 && L > 32) {
        const long long waves = 8ll * device_cu_count();
        const long long per_unit = units * decay_waves(D, SP);
        long long want = (waves + per_unit - 1) / per_unit;
        const long long maxseg = (L + 31) / 32;
        if (want > maxseg) want = maxseg;
        nseg = want < 1 ? 1 : (int)want;
        while (nseg > 1 && (size_t)units * (nseg - 1) * sf_bytes > (size_t(512) << 20)) nseg = (nseg + 1) / 2;
        if (nseg > 1) {
            seg_len = ((L + nseg - 1) / nseg + 15) / 16 * 16;
            nseg = (L + seg_len - 1) / seg_len;
        }
        if (nseg <= 1) {
            nseg = 1;
            seg_len = L;
        }
    }
    dp->nseg = nseg;
    dp->seg_len = seg_len;
    dp->off_summ = align_up(dp->pl.total);
    // sub-block schedules: at most one per head
    const size_t HL = (size_t)(p->H > 0 ? p->H : 0) * L;
    dp->off_gmap = dp->off_summ + align_up((size_t)units * (nseg - 1) * sf_bytes);
    dp->off_glen = dp->off_gmap + align_up((size_t)(p->H > 0 ? p->H : 0) * sizeof(int));
    dp->off_gE = dp->off_glen + align_up(HL * sizeof(int));
    dp->off_gB = dp->off_gE + align_up(HL * SP * sizeof(float));
    dp->total = dp->off_gB + align_up(HL * SP * sizeof(float));
}

// Backward: the one-unit tables (conj_tab = 0, score scale folded into A | B), then the
// forward and adjoint summaries of the segments.  A sequence is cut into segments until the
// main pass has a workgroup per compute unit (the summaries cost one extra pass over every
// segment but the first, so no more are taken).
struct BwdPlan {
    Plan pl;
    int nseg, cps;
    int nbk, cpb;  // summary blocks per sequence and chunks per block
    size_t off_fsum, off_asum, total;
};

bla_status check_backward_shape(const bla_params* p)
{
    bla_status st = check_shape(p, true);
    if (st != BLA_OK) return st;
    if (p->L < 0) return BLA_ERR_INVALID_ARG;
    if (p->phase_anchor != 0) return BLA_ERR_UNSUPPORTED;
    if (p->chunk != 0 && p->chunk != kChunk) return BLA_ERR_UNSUPPORTED;  // the backward runs 64-token chunks
    if (!backward_supported(p->io_dtype == BLA_BF16, p->d_k, pad_modes(p->M), pad_slots(p->S)))
        return BLA_ERR_UNSUPPORTED;
    return BLA_OK;
}

void make_bwd_plan(const bla_params* p, BwdPlan* bp)
{
    make_plan(p, false, &bp->pl);
    Plan& pl = bp->pl;
    pl.pair = 0;
    pl.upw = 1;
    const long long units = (long long)p->B * p->H;
    int nseg = 1;
    const long long cus = device_cu_count();
    if (units > 0 && pl.nch > 1) {
        if (units < cus) {
            long long want = cus / units;
            if (want > pl.nch) want = pl.nch;
            nseg = want < 1 ? 1 : (int)want;
        }
    }
    int cps = pl.nch > 0 ? (pl.nch + nseg - 1) / nseg : 1;
    nseg = pl.nch > 0 ? (pl.nch + cps - 1) / cps : 1;
    bp->nseg = nseg;
    bp->cps = cps;
    // Summary blocks (bf16 kernels): the adjoint summaries cover every segment but the first,
    // (nseg - 1) units of work per sequence, so with few segments that pass would leave compute
    // units idle.  Each segment is cut into bps blocks of cps / bps chunks (the forward and
    // adjoint summaries are taken per block and combined block by block) until the pass has
    // a workgroup per compute unit; the last, possibly shorter, segment must still reach its
    // last block.  The float32 kernels take one block per segment.
    int bps = 1;
    if (p->io_dtype == BLA_BF16 && nseg > 1) {
        const int last_len = pl.nch - (nseg - 1) * cps;  // chunks of the last segment
        while (units * (nseg - 1) * bps < cus && cps % (2 * bps) == 0 &&
               last_len > (2 * bps - 1) * (cps / (2 * bps)))
            bps *= 2;
    }
    bp->nbk = nseg * bps;
    bp->cpb = cps / bps;
    const size_t unit_bytes = (size_t)4 * pl.MP * pl.D * sizeof(float);
    bp->off_fsum = pl.off_summ;
    bp->off_asum = align_up(bp->off_fsum + (size_t)units * bp->nbk * unit_bytes);
    bp->total = align_up(bp->off_asum + (size_t)units * bp->nbk * unit_bytes);
}

}  // namespace

extern "C" {

const char* bla_status_string(bla_status s)
{
    switch (s) {
    case BLA_OK: return "BLA_OK";
    case BLA_ERR_INVALID_ARG: return "BLA_ERR_INVALID_ARG: invalid argument";
    case BLA_ERR_UNSUPPORTED: return "BLA_ERR_UNSUPPORTED: shape not supported by the library";
    case BLA_ERR_WORKSPACE: return "BLA_ERR_WORKSPACE: workspace missing or too small";
    case BLA_ERR_HIP: return "BLA_ERR_HIP: HIP runtime error";
    }
    return "BLA_ERR_UNKNOWN";
}

bla_status bla_supported(const bla_params* p) { return check_shape(p, false); }

bla_status bla_interp_tables(int32_t M, int32_t S, double T, double* A, double* B, int32_t* theta)
{
    if (M < 1 || S < 1 || !A || !B || !theta || !isfinite(T) || T <= 0.0) return BLA_ERR_INVALID_ARG;
    const double Tc = T < 2.0 * M - 1.0 ? 2.0 * M - 1.0 : T;
    for (int s = 0; s < S; ++s) {
        for (int m = 0; m < M; ++m) {
            const double cm = (m == 0 ? 1.0 : 2.0) / (2.0 * M - 1.0);
            const double ph = 2.0 * M_PI * (double)(((long long)m * s) % S) / (double)S;  // exact m s mod S
            A[(size_t)s * M + m] = cm * cos(ph);
            B[(size_t)s * M + m] = cm * sin(ph);
        }
        theta[s] = (int32_t)rint((double)s * Tc / (double)S);
    }
    return BLA_OK;
}

size_t bla_workspace_size(const bla_params* p)
{
    if (check_shape(p, false) != BLA_OK) return 0;
    Plan pl;
    make_plan(p, false, &pl);
    return pl.total;
}

size_t bla_step_workspace_size(const bla_params* p)
{
    if (check_shape(p, true) != BLA_OK) return 0;
    Plan pl;
    make_plan(p, true, &pl);
    return pl.total;
}

// in_strides / out_strides: {batch, head, token} element strides of q, k, v and of o
// (nullable: contiguous [B, H, L, d]).
static bla_status forward_impl(const bla_params* p, const double* T, const void* q, const void* k,
                               const void* v, const long long* in_strides, const float* state_k_in,
                               const float* state_v_in, void* o, const long long* out_strides,
                               float* state_k_out, float* state_v_out, void* workspace,
                               size_t workspace_bytes, void* stream, void* const* events)
{
    bla_status st = check_shape(p, false);
    if (st != BLA_OK) return st;
    if ((st = check_periods(p, T)) != BLA_OK) return st;
    const long long units = (long long)p->B * p->H;
    if (units == 0) return BLA_OK;
    const long long Ld = (long long)p->L * p->d_k;
    const long long contiguous[3] = {(long long)p->H * Ld, Ld, p->d_k};
    const long long* si = in_strides ? in_strides : contiguous;
    const long long* so = out_strides ? out_strides : contiguous;
    for (int i = 0; i < 3; ++i)
        if (si[i] < 0 || so[i] < 0 || si[i] % 8 || so[i] % 8) return BLA_ERR_INVALID_ARG;
    if (si[2] < p->d_k || so[2] < p->d_k || si[2] > INT32_MAX || so[2] > INT32_MAX) return BLA_ERR_INVALID_ARG;
    if (p->L > 0) {
        if (!q || !k || !v || !o) return BLA_ERR_INVALID_ARG;
        if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return BLA_ERR_INVALID_ARG;
    }
    const float* sptr[4] = {state_k_in, state_v_in, state_k_out, state_v_out};
    for (int i = 0; i < 4; ++i)
        if (sptr[i] && !aligned16(sptr[i])) return BLA_ERR_INVALID_ARG;
    if ((state_k_out && state_k_out == state_k_in) || (state_v_out && state_v_out == state_v_in))
        return BLA_ERR_INVALID_ARG;
    Plan pl;
    make_plan(p, false, &pl);
    if (!workspace || workspace_bytes < pl.total || !aligned16(workspace)) return BLA_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const size_t n_state = (size_t)units * 2 * p->M * p->d_k;

    if (p->L == 0) {
        if (launch_state_copy(state_k_in, state_k_out, n_state, s) != hipSuccess) return BLA_ERR_HIP;
        if (launch_state_copy(state_v_in, state_v_out, n_state, s) != hipSuccess) return BLA_ERR_HIP;
        return BLA_OK;
    }
    auto mark = [&](int i) -> bool {
        return !events || !events[i] || hipEventRecord((hipEvent_t)events[i], s) == hipSuccess;
    };
    if (!mark(0)) return BLA_ERR_HIP;
    if ((st = build_tables(pl, T, ws, s, false, p->reuse_tables)) != BLA_OK) return st;
    if (!mark(1)) return BLA_ERR_HIP;

    FwdArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.sk_in = state_k_in;
    a.sv_in = state_v_in;
    a.sk_out = state_k_out;
    a.sv_out = state_v_out;
    a.E32 = (const float*)(ws + pl.off_E32);
    a.EbarT = ws + pl.off_EbarT;
    a.ErevT = ws + pl.off_ErevT;
    a.Etab = ws + pl.off_Etab;
    a.ABs = ws + pl.off_ABs;
    a.ABm = ws + pl.off_ABm;
    if (pl.fragtab) {
        a.fABs = ws + pl.off_fABs;
        a.fABm = ws + pl.off_fABm;
        a.fEtab = ws + pl.off_fEtab;
        a.fEbar = ws + pl.off_fEbar;
        a.fErev = ws + pl.off_fErev;
        a.fTw = ws + pl.off_fTw;
    }
    a.theta = (const int*)(ws + pl.off_theta);
    a.summ = (float*)(ws + pl.off_summ);
    a.carry = (float*)(ws + pl.off_carry);
    a.rotblk = (const float*)(ws + pl.off_rotblk);
    a.rperiod = (const double*)(ws + pl.off_rperiod);
    a.anchor = pl.anchor;
    a.B = pl.B;
    a.H = pl.H;
    a.L = pl.L;
    a.M = pl.M;
    a.C = pl.C;
    a.nch = pl.nch;
    a.nseg = pl.nseg;
    a.cps = pl.cps;
    a.cpb = pl.cpb;
    a.nbs = pl.nbs;
    a.t0 = pl.t0;
    a.scale = pl.scale;
    a.in_b = si[0];
    a.in_h = si[1];
    a.in_t = (int)si[2];
    a.out_b = so[0];
    a.out_h = so[1];
    a.out_t = (int)so[2];
    if (pl.nseg > 1 && launch_summary(pl, a, s) != hipSuccess) return BLA_ERR_HIP;
    if (!mark(2)) return BLA_ERR_HIP;
    if (pl.nseg > 1 && !pl.pair && launch_scan(pl, a, s) != hipSuccess) return BLA_ERR_HIP;
    if (!mark(3)) return BLA_ERR_HIP;
    if (launch_forward(pl, a, s) != hipSuccess) return BLA_ERR_HIP;
    if (!mark(4)) return BLA_ERR_HIP;
    return BLA_OK;
}

bla_status bla_forward(const bla_params* p, const double* T, const void* q, const void* k,
                       const void* v, const float* state_k_in, const float* state_v_in, void* o,
                       float* state_k_out, float* state_v_out, void* workspace,
                       size_t workspace_bytes, void* stream)
{
    return forward_impl(p, T, q, k, v, nullptr, state_k_in, state_v_in, o, nullptr, state_k_out, state_v_out,
                        workspace, workspace_bytes, stream, nullptr);
}

bla_status bla_forward_timed(const bla_params* p, const double* T, const void* q, const void* k,
                             const void* v, const float* state_k_in, const float* state_v_in, void* o,
                             float* state_k_out, float* state_v_out, void* workspace,
                             size_t workspace_bytes, void* stream, void* const* events)
{
    return forward_impl(p, T, q, k, v, nullptr, state_k_in, state_v_in, o, nullptr, state_k_out, state_v_out,
                        workspace, workspace_bytes, stream, events);
}

bla_status bla_step(const bla_params* p, const double* T, const void* q, const void* k,
                    const void* v, const int64_t* pos, float* state_k, float* state_v, void* o,
                    void* workspace, size_t workspace_bytes, void* stream)
{
    bla_status st = check_shape(p, true);
    if (st != BLA_OK) return st;
    if ((st = check_periods(p, T)) != BLA_OK) return st;
    const long long units = (long long)p->B * p->H;
    if (units == 0) return BLA_OK;
    if (!q || !k || !v || !o || !state_k || !state_v) return BLA_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(state_k) ||
        !aligned16(state_v))
        return BLA_ERR_INVALID_ARG;
    if (pos && ((uintptr_t)pos & 7u)) return BLA_ERR_INVALID_ARG;
    Plan pl;
    make_plan(p, true, &pl);
    if (!workspace || workspace_bytes < pl.total || !aligned16(workspace)) return BLA_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    if ((st = build_tables(pl, T, ws, s, true, p->reuse_tables)) != BLA_OK) return st;
    StepArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.pos = pos;
    a.sk = state_k;
    a.sv = state_v;
    a.E32 = (const float*)(ws + pl.off_E32);
    a.trig = (const float*)(ws + pl.off_trig);
    a.theta = (const int*)(ws + pl.off_theta);
    a.rperiod = (const double*)(ws + pl.off_rperiod);
    a.anchor = pl.anchor;
    a.B = pl.B;
    a.H = pl.H;
    a.M = pl.M;
    a.S = pl.S;
    a.SP = pl.SP;
    a.t0 = pl.t0;
    a.scale = pl.scale;
    if (launch_step(pl, a, s) != hipSuccess) return BLA_ERR_HIP;
    return BLA_OK;
}

// ---------------------------------------------------------------- state-decay form (Sec. 3.4)

size_t bla_decay_workspace_size(const bla_params* p)
{
    if (check_shape(p, true) != BLA_OK || p->L < 0) return 0;
    DecayPlan dp;
    make_decay_plan(p, &dp);
    return dp.total;
}

static bla_status decay_forward_impl(const bla_params* p, const double* T, const void* q, const void* k,
                                     const void* v, const float* slot_k_in, const float* slot_v_in, void* o,
                                     float* slot_k_out, float* slot_v_out, void* workspace,
                                     size_t workspace_bytes, void* stream, void* const* events)
{
    bla_status st = check_shape(p, true);
    if (st != BLA_OK) return st;
    if (p->L < 0) return BLA_ERR_INVALID_ARG;
    if ((st = check_periods(p, T)) != BLA_OK) return st;
    const long long units = (long long)p->B * p->H;
    if (units == 0) return BLA_OK;
    if (p->L > 0) {
        if (!q || !k || !v || !o) return BLA_ERR_INVALID_ARG;
        if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return BLA_ERR_INVALID_ARG;
    }
    const float* sptr[4] = {slot_k_in, slot_v_in, slot_k_out, slot_v_out};
    for (int i = 0; i < 4; ++i)
        if (sptr[i] && !aligned16(sptr[i])) return BLA_ERR_INVALID_ARG;
    if ((slot_k_out && slot_k_out == slot_k_in) || (slot_v_out && slot_v_out == slot_v_in))
        return BLA_ERR_INVALID_ARG;
    DecayPlan dp;
    make_decay_plan(p, &dp);
    const Plan& pl = dp.pl;
    if (!workspace || workspace_bytes < dp.total || !aligned16(workspace)) return BLA_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    if (p->L == 0) {
        const size_t n = (size_t)units * p->S * p->d_k;
        if (launch_state_copy(slot_k_in, slot_k_out, n, s) != hipSuccess) return BLA_ERR_HIP;
        if (launch_state_copy(slot_v_in, slot_v_out, n, s) != hipSuccess) return BLA_ERR_HIP;
        return BLA_OK;
    }
    auto mark = [&](int i) -> bool {
        return !events || !events[i] || hipEventRecord((hipEvent_t)events[i], s) == hipSuccess;
    };
    if (!mark(0)) return BLA_ERR_HIP;
    if ((st = build_tables(pl, T, ws, s, true, p->reuse_tables)) != BLA_OK) return st;
    DecayArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.sk_in = slot_k_in;
    a.sv_in = slot_v_in;
    a.sk_out = slot_k_out;
    a.sv_out = slot_v_out;
    a.theta = (const int*)(ws + pl.off_theta);
    a.period = (const double*)(ws + pl.off_period);
    a.rperiod = (const double*)(ws + pl.off_rperiod);
    a.summ = (float*)(ws + dp.off_summ);
    a.gE = (const float*)(ws + dp.off_gE);
    a.gB = (const float*)(ws + dp.off_gB);
    a.glen = (const int*)(ws + dp.off_glen);
    a.gmap = (const int*)(ws + dp.off_gmap);
    a.B = p->B;
    a.H = p->H;
    a.L = p->L;
    a.M = p->M;
    a.S = p->S;
    a.nseg = dp.nseg;
    a.seg_len = dp.seg_len;
    a.t0 = p->t0;
    a.scale = pl.scale;
    // sub-block schedules: one per distinct clamped period within each group of heads
    {
        int ubase = 0;
        for (int h0 = 0; h0 < p->H; h0 += kMaxHeadsPerTableLaunch) {
            GateArgs g;
            memset(&g, 0, sizeof(g));
            g.gE = (float*)(ws + dp.off_gE);
            g.gB = (float*)(ws + dp.off_gB);
            g.glen = (int*)(ws + dp.off_glen);
            g.gmap = (int*)(ws + dp.off_gmap);
            g.L = p->L;
            g.SP = pl.SP;
            g.S = p->S;
            g.M = p->M;
            g.h0 = h0;
            g.nh = p->H - h0 < kMaxHeadsPerTableLaunch ? p->H - h0 : kMaxHeadsPerTableLaunch;
            g.ubase = ubase;
            g.t0 = p->t0;
            g.rS = 1.0 / (double)p->S;
            double per[kMaxHeadsPerTableLaunch];
            for (int i = 0; i < g.nh; ++i) {
                const double tmin = 2.0 * p->M - 1.0;
                const double Tp = T[h0 + i] < tmin ? tmin : T[h0 + i];  // clamped as the tables kernel does
                int u = 0;
                while (u < g.nu && per[u] != Tp) ++u;
                if (u == g.nu) {
                    per[g.nu] = Tp;
                    g.rT[g.nu] = 1.0 / Tp;
                    ++g.nu;
                }
                g.map[i] = ubase + u;
            }
            if (launch_decay_gates(g, s) != hipSuccess) return BLA_ERR_HIP;
            ubase += g.nu;
        }
    }
    if (!mark(1)) return BLA_ERR_HIP;
    if (launch_decay_forward(pl.bf16, pl.D, pl.SP, a, s, events ? events + 2 : nullptr) != hipSuccess)
        return BLA_ERR_HIP;
    return BLA_OK;
}

bla_status bla_decay_forward(const bla_params* p, const double* T, const void* q, const void* k,
                             const void* v, const float* slot_k_in, const float* slot_v_in, void* o,
                             float* slot_k_out, float* slot_v_out, void* workspace, size_t workspace_bytes,
                             void* stream)
{
    return decay_forward_impl(p, T, q, k, v, slot_k_in, slot_v_in, o, slot_k_out, slot_v_out, workspace,
                              workspace_bytes, stream, nullptr);
}

bla_status bla_decay_forward_timed(const bla_params* p, const double* T, const void* q, const void* k,
                                   const void* v, const float* slot_k_in, const float* slot_v_in, void* o,
                                   float* slot_k_out, float* slot_v_out, void* workspace,
                                   size_t workspace_bytes, void* stream, void* const* events)
{
    return decay_forward_impl(p, T, q, k, v, slot_k_in, slot_v_in, o, slot_k_out, slot_v_out, workspace,
                              workspace_bytes, stream, events);
}

bla_status bla_decay_step(const bla_params* p, const double* T, const void* q, const void* k,
                          const void* v, const int64_t* pos, float* slot_k, float* slot_v, void* o,
                          void* workspace, size_t workspace_bytes, void* stream)
{
    bla_status st = check_shape(p, true);
    if (st != BLA_OK) return st;
    if ((st = check_periods(p, T)) != BLA_OK) return st;
    const long long units = (long long)p->B * p->H;
    if (units == 0) return BLA_OK;
    if (!q || !k || !v || !o || !slot_k || !slot_v) return BLA_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(slot_k) ||
        !aligned16(slot_v))
        return BLA_ERR_INVALID_ARG;
    if (pos && ((uintptr_t)pos & 7u)) return BLA_ERR_INVALID_ARG;
    Plan pl;
    make_plan(p, true, &pl);
    if (!workspace || workspace_bytes < pl.total || !aligned16(workspace)) return BLA_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    if ((st = build_tables(pl, T, ws, s, true, p->reuse_tables)) != BLA_OK) return st;
    DecayStepArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.pos = pos;
    a.sk = slot_k;
    a.sv = slot_v;
    a.theta = (const int*)(ws + pl.off_theta);
    a.rperiod = (const double*)(ws + pl.off_rperiod);
    a.B = p->B;
    a.H = p->H;
    a.M = p->M;
    a.S = p->S;
    a.t0 = p->t0;
    a.scale = pl.scale;
    if (launch_decay_step(pl.bf16, pl.D, pl.SP, a, s) != hipSuccess) return BLA_ERR_HIP;
    return BLA_OK;
}

size_t bla_backward_workspace_size(const bla_params* p)
{
    if (check_backward_shape(p) != BLA_OK) return 0;
    BwdPlan bp;
    make_bwd_plan(p, &bp);
    return bp.total;
}

static bla_status backward_impl(const bla_params* p, const double* T, const void* q, const void* k,
                                const void* v, const void* dO, const float* state_k_in,
                                const float* state_v_in, const float* dstate_k_out,
                                const float* dstate_v_out, void* dq, void* dk, void* dv,
                                float* dstate_k_in, float* dstate_v_in, void* workspace,
                                size_t workspace_bytes, void* stream, void* const* events)
{
    bla_status st = check_backward_shape(p);
    if (st != BLA_OK) return st;
    if ((st = check_periods(p, T)) != BLA_OK) return st;
    const long long units = (long long)p->B * p->H;
    if (units == 0) return BLA_OK;
    if (p->L > 0) {
        const void* t[7] = {q, k, v, dO, dq, dk, dv};
        for (int i = 0; i < 7; ++i)
            if (!t[i] || !aligned16(t[i])) return BLA_ERR_INVALID_ARG;
    }
    const float* sptr[6] = {state_k_in, state_v_in, dstate_k_out, dstate_v_out, dstate_k_in, dstate_v_in};
    for (int i = 0; i < 6; ++i)
        if (sptr[i] && !aligned16(sptr[i])) return BLA_ERR_INVALID_ARG;
    if ((dstate_k_in && (dstate_k_in == dstate_k_out || dstate_k_in == state_k_in)) ||
        (dstate_v_in && (dstate_v_in == dstate_v_out || dstate_v_in == state_v_in)))
        return BLA_ERR_INVALID_ARG;
    BwdPlan bp;
    make_bwd_plan(p, &bp);
    if (!workspace || workspace_bytes < bp.total || !aligned16(workspace)) return BLA_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const Plan& pl = bp.pl;
    const size_t n_state = (size_t)units * 2 * p->M * p->d_k;
    if (p->L == 0) {
        // no tokens: the input states are the final states
        if (launch_state_copy(dstate_k_out, dstate_k_in, n_state, s) != hipSuccess) return BLA_ERR_HIP;
        if (launch_state_copy(dstate_v_out, dstate_v_in, n_state, s) != hipSuccess) return BLA_ERR_HIP;
        return BLA_OK;
    }
    auto mark = [&](int i) -> bool {
        return !events || !events[i] || hipEventRecord((hipEvent_t)events[i], s) == hipSuccess;
    };
    if (!mark(0)) return BLA_ERR_HIP;
    if ((st = build_tables(pl, T, ws, s, false, p->reuse_tables)) != BLA_OK) return st;
    if (!mark(1)) return BLA_ERR_HIP;
    BwdArgs a;
    memset(&a, 0, sizeof(a));
    a.q = q;
    a.k = k;
    a.v = v;
    a.dO = dO;
    a.sk_in = state_k_in;
    a.sv_in = state_v_in;
    a.gk_out = dstate_k_out;
    a.gv_out = dstate_v_out;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.gk_in = dstate_k_in;
    a.gv_in = dstate_v_in;
    a.E32 = (const float*)(ws + pl.off_E32);
    a.EbarT = ws + pl.off_EbarT;
    a.ErevT = ws + pl.off_ErevT;
    a.Etab = ws + pl.off_Etab;
    a.ABs = ws + pl.off_ABs;
    a.ABm = ws + pl.off_ABm;
    a.theta = (const int*)(ws + pl.off_theta);
    a.rperiod = (const double*)(ws + pl.off_rperiod);
    a.fsum = (float*)(ws + bp.off_fsum);
    a.asum = (float*)(ws + bp.off_asum);
    a.B = p->B;
    a.H = p->H;
    a.L = p->L;
    a.M = p->M;
    a.nch = pl.nch;
    a.nseg = bp.nseg;
    a.cps = bp.cps;
    a.nbk = bp.nbk;
    a.cpb = bp.cpb;
    a.t0 = p->t0;
    a.scale = pl.scale;
    void* ev3[3] = {events ? events[2] : nullptr, events ? events[3] : nullptr, events ? events[4] : nullptr};
    if (launch_backward(pl.bf16, pl.D, pl.MP, pl.SP, a, s, ev3) != hipSuccess) return BLA_ERR_HIP;
    return BLA_OK;
}

bla_status bla_backward(const bla_params* p, const double* T, const void* q, const void* k, const void* v,
                        const void* dO, const float* state_k_in, const float* state_v_in,
                        const float* dstate_k_out, const float* dstate_v_out, void* dq, void* dk, void* dv,
                        float* dstate_k_in, float* dstate_v_in, void* workspace, size_t workspace_bytes,
                        void* stream)
{
    return backward_impl(p, T, q, k, v, dO, state_k_in, state_v_in, dstate_k_out, dstate_v_out, dq, dk, dv,
                         dstate_k_in, dstate_v_in, workspace, workspace_bytes, stream, nullptr);
}

bla_status bla_backward_timed(const bla_params* p, const double* T, const void* q, const void* k,
                              const void* v, const void* dO, const float* state_k_in, const float* state_v_in,
                              const float* dstate_k_out, const float* dstate_v_out, void* dq, void* dk,
                              void* dv, float* dstate_k_in, float* dstate_v_in, void* workspace,
                              size_t workspace_bytes, void* stream, void* const* events)
{
    return backward_impl(p, T, q, k, v, dO, state_k_in, state_v_in, dstate_k_out, dstate_v_out, dq, dk, dv,
                         dstate_k_in, dstate_v_in, workspace, workspace_bytes, stream, events);
}

}  // extern "C"

namespace bla {

bla_status forward_strided(const bla_params* p, const double* T, const void* q, const void* k, const void* v,
                           const long long* in_strides, const float* state_k_in, const float* state_v_in, void* o,
                           const long long* out_strides, float* state_k_out, float* state_v_out, void* workspace,
                           size_t workspace_bytes, void* stream, void* const* events)
{
    return forward_impl(p, T, q, k, v, in_strides, state_k_in, state_v_in, o, out_strides, state_k_out,
                        state_v_out, workspace, workspace_bytes, stream, events);
}

}  // namespace bla
