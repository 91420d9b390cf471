// C-ABI entry points: validation, workspace carving and kernel launches on
// the caller's stream.  See include/convbwd.h for the contract.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstring>
#include <mutex>

#include "../../include/convbwd.h"
#include "kernels.hpp"
#include "plan.hpp"
#include "reduce.hpp"

using namespace cbw;

namespace {

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Profiling events per op family (0 = data gradient, 1 = weight gradient,
// 2 = forward).
thread_local hipEvent_t g_prof[3][2] = {{nullptr, nullptr}, {nullptr, nullptr}, {nullptr, nullptr}};

ProfEvents prof_events(int fam)
{
    ProfEvents ev;
    ev.start = g_prof[fam][0];
    ev.stop = g_prof[fam][1];
    return ev;
}

int hip_status(hipError_t e)
{
    if (e == hipSuccess) return CBW_OK;
    (void)hipGetLastError();
    return CBW_ERR_HIP;
}

template <typename T>
T* at(void* ws, const Region& r) { return reinterpret_cast<T*>(static_cast<char*>(ws) + r.off); }

bool tiles_consistent()
{
    static_assert(kDataMaxSplit >= 1, "split bound");
    if (data_split(1, 1 << 20, kDataSlots, kDataMaxSplit) != host_data_split(1, 1 << 20)) return false;
    for (int t = 0; t < kDataTileCount; ++t)
        if (data_tile_channels(t) != kDataTiles[t].bm || data_tile_pixels(t) != kDataTiles[t].bn) return false;
    if (data_rows_segment() != kDataRowsSegment) return false;
    if (data_pw_waves_per_group() != kDataPwWaves) return false;
    return weight_tile_channels() == kWeightTileC && weight_tile_k() == kWeightTileK &&
           compact_block_pixels() == kCompactBlock && weight_chunk(CBW_BF16) == weight_chunk_px(CBW_BF16) &&
           weight_chunk(CBW_F32) == weight_chunk_px(CBW_F32);
}

int check_ws(const void* ws, size_t ws_bytes, size_t need)
{
    if (need > 0 && ws == nullptr) return CBW_ERR_WORKSPACE;
    if (ws_bytes < need) return CBW_ERR_WORKSPACE;
    if (!aligned16(ws)) return CBW_ERR_UNSUPPORTED;
    return CBW_OK;
}

DataParams data_params(const cbw_conv_desc* d, const void* dY, const void* wt, void* dX, int64_t npix,
                       int groups)
{
    DataParams p{};
    p.dy = dY;
    p.wt = wt;
    p.dx = dX;
    p.N = d->N; p.H = d->H; p.W = d->W; p.C = d->C; p.K = d->K; p.R = d->R; p.S = d->S;
    p.P = d->P; p.Q = d->Q;
    p.stride_h = d->stride_h; p.stride_w = d->stride_w; p.pad_h = d->pad_h; p.pad_w = d->pad_w;
    p.npix = (int)npix;
    p.ctiles = groups;
    p.div_w = make_fastdiv((uint32_t)d->W);
    p.div_h = make_fastdiv((uint32_t)d->H);
    const int64_t esz = elem_bytes(d->dtype);
    p.dy_bytes = (uint32_t)((int64_t)d->N * d->P * d->Q * d->K * esz);
    p.wt_bytes = (uint32_t)((int64_t)d->R * d->S * d->C * d->K * esz);
    p.dx_bytes = (uint32_t)(npix * d->C * esz);
    return p;
}

// Kernel parameters of the data gradient on NHWC tensors (dY, dX, x_mask
// already in NHWC order), from a validated plan.
void data_gemm_params(const cbw_conv_desc* desc, const DataPlan& plan, const void* dY, const void* wt,
                      const uint32_t* x_mask, void* dX, void* ws, bool gather, bool no_split, DataParams* out,
                      CompactParams* cpo)
{
    DataParams p = data_params(desc, dY, wt, dX, plan.npix, plan.groups);
    p.tile = plan.tile;
    p.mask = x_mask;
    p.ptiles = plan.ptiles;
    p.brows = plan.brows;
    p.nslots = kDataSlots;
    p.smax = no_split ? 1 : kDataMaxSplit;
    p.split = plan.split;   // gather mode: the split of its dense tiles, which it checks on the device
    p.partial = plan.partial.bytes ? at<float>(ws, plan.partial) : nullptr;
    CompactParams cp{};
    if (gather) {
        cp.mask = x_mask;
        cp.blk_counts = at<int32_t>(ws, plan.blk_counts);
        cp.dead_flags = at<int32_t>(ws, plan.dead_flags);
        cp.dx = dX;
        cp.npix = (int)plan.npix;
        cp.C = desc->C;
        cp.G = plan.bm;
        cp.groups = plan.groups;
        cp.nblk = plan.nblk;
        cp.elem_bytes = elem_bytes(desc->dtype);
        p.blk_counts = cp.blk_counts;
        p.nblk = plan.nblk;
        p.lists = at<int32_t>(ws, plan.lists);
        p.counts = at<int32_t>(ws, plan.counts);
        p.dead_flags = cp.dead_flags;
    }
    *out = p;
    *cpo = cp;
}

// Kernel parameters of the row-window data gradient (NHWC tensors).
DataRowsParams data_rows_params(const cbw_conv_desc* d, const DataPlan& plan, const void* dY, const void* wt,
                                const uint32_t* x_mask, void* dX, void* ws, bool skip)
{
    DataRowsParams p{};
    p.dy = dY;
    p.wt = wt;
    p.dx = dX;
    p.mask = x_mask;
    p.row_counts = at<int32_t>(ws, plan.row_counts);
    p.N = d->N; p.H = d->H; p.W = d->W; p.P = d->P; p.Q = d->Q;
    p.pad_h = d->pad_h; p.pad_w = d->pad_w;
    p.nseg = plan.rows_nseg;
    p.rows_per_strip = plan.rows_per_strip;
    p.nrows = d->N * d->H;
    p.skip = x_mask && skip ? 1 : 0;
    const int64_t esz = elem_bytes(d->dtype);
    p.dy_bytes = (uint32_t)((int64_t)d->N * d->P * d->Q * d->K * esz);
    p.dx_bytes = (uint32_t)(plan.npix * d->C * esz);
    p.mask_bytes = (uint32_t)((plan.npix * d->C + 31) / 32 * 4);
    p.wt_bytes = (uint32_t)((int64_t)d->R * d->S * d->C * d->K * esz);
    p.div_h = make_fastdiv((uint32_t)d->H);
    p.depth = plan.rows_depth;
    p.nslot = plan.rows_depth + 3;
    p.slot_bytes = plan.rows_slot;
    p.mslot_bytes = plan.rows_mslot;
    p.mask_off = p.nslot * p.slot_bytes;
    p.div_nslot = make_fastdiv((uint32_t)p.nslot);
    p.div_nmslot = make_fastdiv((uint32_t)(p.depth + 2));
    return p;
}

// Kernel parameters of the pointwise data gradient (NHWC tensors).
DataPwParams data_pw_params(const cbw_conv_desc* d, const DataPlan& plan, const void* dY, const void* wt,
                            const uint32_t* x_mask, void* dX, void* ws, bool skip)
{
    DataPwParams p{};
    p.dy = dY;
    p.wt = wt;
    p.dx = dX;
    p.mask = x_mask;
    p.counts = at<int32_t>(ws, plan.row_counts);
    p.npix = (int)plan.npix;
    p.C = d->C;
    p.K = d->K;
    p.nblk = (int)((plan.npix + 15) / 16);
    p.bpw = plan.pw_bpw;
    p.skip = x_mask && skip ? 1 : 0;
    const int64_t esz = elem_bytes(d->dtype);
    p.dy_bytes = (uint32_t)(plan.npix * d->K * esz);
    p.dx_bytes = (uint32_t)(plan.npix * d->C * esz);
    p.mask_bytes = (uint32_t)((plan.npix * d->C + 31) / 32 * 4);
    return p;
}

// compaction needs at most kGatherMaxGroups channel groups; wider layers
// keep the footprint select without it
bool data_gathers(const DataPlan& plan, bool masked, uint32_t flags)
{
    return masked && !(flags & CBW_FLAG_NO_SKIP) && plan.groups <= kGatherMaxGroups;
}

// Offset of the weight-gradient part in the workspace of the call that
// computes both gradients: after the masked data gradient's workspace.
int both_offset(const cbw_conv_desc* desc, size_t* off, size_t* total)
{
    DataPlan dp;
    size_t wbytes = 0;
    int st = plan_data(desc, true, &dp);
    if (st != CBW_OK) return st;
    if ((st = weight_ws_bytes(desc, &wbytes)) != CBW_OK) return st;
    *off = (dp.total + 255) & ~(size_t)255;
    *total = *off + wbytes;
    return CBW_OK;
}

// The weight-gradient plan the last call on `workspace` ran (its kernel
// stamps which one into the header), for the readers.
int last_weight_plan(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, WeightPlan* plan,
                     hipStream_t s)
{
    WeightPlan p;
    int st = plan_weight(desc, &p, false);
    if (st != CBW_OK) return st;
    if (!workspace) return CBW_ERR_INVALID_ARG;
    if (workspace_bytes < 256) return CBW_ERR_WORKSPACE;
    int hdr[2] = {0, 0};
    hipError_t e = hipMemcpyAsync(hdr, workspace, sizeof(hdr), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_status(e);
    if ((st = plan_weight(desc, &p, hdr[1] == 1)) != CBW_OK) return st;
    if (workspace_bytes < p.total) return CBW_ERR_WORKSPACE;
    *plan = p;
    return CBW_OK;
}

int run_bwd_data(const cbw_conv_desc* desc, const void* dY, const void* W, const uint32_t* x_mask, void* dX,
                 void* ws, size_t ws_bytes, uint32_t flags, void* stream, bool masked, bool no_split = false)
{
    DataPlan plan;
    int st = plan_data(desc, masked, &plan, no_split);
    if (st != CBW_OK) return st;
    if (!dY || !W || !dX || (masked && !x_mask)) return CBW_ERR_INVALID_ARG;
    if (!aligned16(dY) || !aligned16(W) || !aligned16(dX) || (masked && !aligned16(x_mask)))
        return CBW_ERR_UNSUPPORTED;
    if ((st = check_ws(ws, ws_bytes, plan.total)) != CBW_OK) return st;
    if (!tiles_consistent()) return CBW_ERR_UNSUPPORTED;
    hipStream_t s = static_cast<hipStream_t>(stream);

    const bool gather = data_gathers(plan, masked, flags);
    const int mode = !masked ? MODE_DENSE : (gather ? MODE_GATHER : MODE_SELECT);
    hipError_t e;
    void* dX_out = dX;
    if (desc->act_layout == CBW_NCHW) {
        // the kernels read an NHWC copy of dY (and an NHWC-order footprint)
        // and write an NHWC dX, transposed into the caller's dX at the end
        void* tdy = at<void>(ws, plan.t_dy);
        if ((e = launch_transpose(desc->dtype, dY, tdy, desc->N, desc->K, desc->P * desc->Q, s)) != hipSuccess)
            return hip_status(e);
        dY = tdy;
        dX = at<void>(ws, plan.t_dx);
        if (masked) {
            uint32_t* t = at<uint32_t>(ws, plan.t_mask);
            if ((e = launch_bits_nchw_to_nhwc(x_mask, t, desc->N, desc->C, desc->H * desc->W, s)) != hipSuccess)
                return hip_status(e);
            x_mask = t;
        }
    }
    int* header = at<int>(ws, plan.header);
    void* wt = at<void>(ws, plan.wt);
    if (plan.rows) {
        e = launch_data_prep(desc->dtype, W, wt, desc->K, desc->C, desc->R * desc->S, desc->w_layout == CBW_KRSC,
                             header, MODE_ROWS, nullptr, s);
        if (e != hipSuccess) return hip_status(e);
        const DataRowsParams rp = data_rows_params(desc, plan, dY, wt, masked ? x_mask : nullptr, dX, ws,
                                                   !(flags & CBW_FLAG_NO_SKIP));
        if ((e = launch_bwd_data_rows(rp, plan.rows_grid, plan.rows_nbw, s, prof_events(0))) != hipSuccess)
            return hip_status(e);
    } else if (plan.pw) {
        e = launch_data_prep(desc->dtype, W, wt, desc->K, desc->C, 1, desc->w_layout == CBW_KRSC, header, MODE_PW,
                             nullptr, s);
        if (e != hipSuccess) return hip_status(e);
        const DataPwParams pp = data_pw_params(desc, plan, dY, wt, masked ? x_mask : nullptr, dX, ws,
                                               !(flags & CBW_FLAG_NO_SKIP));
        if ((e = launch_bwd_data_pw(pp, plan.pw_grid, s, prof_events(0))) != hipSuccess) return hip_status(e);
    } else {
        DataParams p;
        CompactParams cp;
        data_gemm_params(desc, plan, dY, wt, x_mask, dX, ws, gather, no_split, &p, &cp);
        e = launch_data_prep(desc->dtype, W, wt, desc->K, desc->C, desc->R * desc->S, desc->w_layout == CBW_KRSC,
                             header, mode, gather ? &cp : nullptr, s);
        if (e != hipSuccess) return hip_status(e);
        if ((e = launch_bwd_data(desc->dtype, mode, p, s, prof_events(0))) != hipSuccess) return hip_status(e);
    }
    if (dX != dX_out)
        e = launch_transpose(desc->dtype, dX, dX_out, desc->N, desc->H * desc->W, desc->C, s);
    return hip_status(e);
}

int run_fwd(const cbw_conv_desc* desc, const void* X, const void* W, void* Y, uint32_t* y_mask, void* ws,
            size_t ws_bytes, void* stream)
{
    cbw_conv_desc vd;
    int st = fwd_as_data_desc(desc, &vd);
    if (st != CBW_OK) return st;
    DataPlan plan;
    if ((st = plan_data(&vd, false, &plan, false, false)) != CBW_OK) return st;
    if (!X || !W || !Y) return CBW_ERR_INVALID_ARG;
    if (!aligned16(X) || !aligned16(W) || !aligned16(Y) || (y_mask && !aligned16(y_mask)))
        return CBW_ERR_UNSUPPORTED;
    if ((st = check_ws(ws, ws_bytes, plan.total)) != CBW_OK) return st;
    if (!tiles_consistent()) return CBW_ERR_UNSUPPORTED;
    hipStream_t s = static_cast<hipStream_t>(stream);

    int* header = at<int>(ws, plan.header);
    void* wt = at<void>(ws, plan.wt);
    DataParams p = data_params(&vd, X, wt, Y, plan.npix, plan.groups);
    p.tile = plan.tile;
    p.ptiles = plan.ptiles;
    p.brows = plan.brows;
    p.nslots = kDataSlots;
    p.smax = kDataMaxSplit;
    p.split = plan.split;
    p.partial = plan.partial.bytes ? at<float>(ws, plan.partial) : nullptr;
    p.out_mask = y_mask;
    // footprint words are assembled whole in the GEMM epilogue when the
    // output channel count is a multiple of 32 and nothing is split;
    // otherwise they are OR-ed in and must start cleared
    const int64_t words = ((int64_t)desc->N * desc->P * desc->Q * desc->K + 31) / 32;
    const bool clear = y_mask && (desc->K % 32 != 0 || plan.split > 1);
    hipError_t e = launch_fwd_prep(desc->dtype, W, wt, desc->K, desc->C, desc->R, desc->S,
                                   desc->w_layout == CBW_KRSC, header, clear ? y_mask : nullptr,
                                   clear ? words : 0, s);
    if (e != hipSuccess) return hip_status(e);
    return hip_status(launch_bwd_data(desc->dtype, MODE_FWD, p, s, prof_events(2)));
}

// Built-in scratch of conv_bwd_data_masked_noalloc: the masked data
// gradient's workspace (filter transform, compaction counts and lists) for
// callers that cannot allocate.  Each GPU the library runs on holds its own
// copy until the process ends.  Host code never uses the array's name as an
// address: its device address is looked up once per device
// (hipGetSymbolAddress) and kept in g_scratch_dev.
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of the current device's scratch (looked up on first use).
int scratch_for_current_device(void** out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e);
    if (dev < 0 || dev >= kMaxDevices) return CBW_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(e);
        if (!ptr) return CBW_ERR_HIP;
        g_scratch_dev[dev] = ptr;
    }
    *out = g_scratch_dev[dev];
    return CBW_OK;
}

}  // namespace

extern "C" {

const char* cbw_status_string(int status)
{
    switch (status) {
    case CBW_OK: return "ok";
    case CBW_ERR_INVALID_ARG: return "invalid argument";
    case CBW_ERR_UNSUPPORTED: return "unsupported configuration";
    case CBW_ERR_WORKSPACE: return "workspace missing or too small";
    case CBW_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

int cbw_validate_desc(const cbw_conv_desc* desc) { return validate_desc(desc); }

size_t cbw_mask_words(const cbw_conv_desc* d)
{
    if (validate_desc(d) != CBW_OK) return 0;
    return (size_t)(((int64_t)d->N * d->C * d->H * d->W + 31) / 32);
}

size_t cbw_dy_mask_words(const cbw_conv_desc* d)
{
    if (validate_desc(d) != CBW_OK) return 0;
    return (size_t)(((int64_t)d->N * d->K * d->P * d->Q + 31) / 32);
}

// Descriptors the per-element data gradient supports.
static int validate_elementwise(const cbw_conv_desc* d)
{
    const int st = require_nhwc(d);
    if (st != CBW_OK) return st;
    if (d->dtype != CBW_BF16 || d->w_layout != CBW_KRSC) return CBW_ERR_UNSUPPORTED;
    if (d->C != 64 && d->C != 128 && d->C != 256 && d->C != 512) return CBW_ERR_UNSUPPORTED;
    if (d->K >= 65536) return CBW_ERR_UNSUPPORTED;   // k is packed in 16 bits
    if (d->R * d->S > 255) return CBW_ERR_UNSUPPORTED;   // the tap is kept in 8 bits
    return CBW_OK;
}

// Workspace of the per-element data gradient: an int32 count per output pixel.
static size_t elementwise_ws(const cbw_conv_desc* d)
{
    return ((size_t)d->N * d->H * d->W * 4 + 255) / 256 * 256;
}

int cbw_data_tiling(const cbw_conv_desc* desc, int32_t* channels, int32_t* capacity, int32_t* rows)
{
    DataPlan p;
    const int st = plan_data(desc, false, &p, false, false);
    if (st != CBW_OK) return st;
    if (channels) *channels = p.bm;
    if (capacity) *capacity = p.bn;
    if (rows) *rows = p.brows;
    return CBW_OK;
}

int cbw_workspace_size(const cbw_conv_desc* desc, int op, size_t* bytes)
{
    if (!bytes) return CBW_ERR_INVALID_ARG;
    int st;
    if (op == CBW_OP_BWD_DATA || op == CBW_OP_BWD_DATA_MASKED) {
        DataPlan p;
        if ((st = plan_data(desc, op == CBW_OP_BWD_DATA_MASKED, &p)) != CBW_OK) return st;
        *bytes = p.total;
        return CBW_OK;
    }
    if (op == CBW_OP_BWD_WEIGHT) return weight_ws_bytes(desc, bytes);
    if (op == CBW_OP_BWD_DATA_ELEMENTWISE) {
        if ((st = validate_elementwise(desc)) != CBW_OK) return st;
        *bytes = elementwise_ws(desc);
        return CBW_OK;
    }
    if (op == CBW_OP_BWD_BOTH) {
        size_t off;
        if ((st = both_offset(desc, &off, bytes)) != CBW_OK) return st;
        return CBW_OK;
    }
    if (op == CBW_OP_FWD) {
        cbw_conv_desc vd;
        DataPlan p;
        if ((st = fwd_as_data_desc(desc, &vd)) != CBW_OK) return st;
        if ((st = plan_data(&vd, false, &p, false, false)) != CBW_OK) return st;
        *bytes = p.total;
        return CBW_OK;
    }
    return CBW_ERR_INVALID_ARG;
}

int cbw_relu_mask_pack(const cbw_conv_desc* desc, const void* X, uint32_t* x_mask, void* stream)
{
    int st = validate_desc(desc);
    if (st != CBW_OK) return st;
    if (!X || !x_mask) return CBW_ERR_INVALID_ARG;
    if (!aligned16(X) || ((uintptr_t)x_mask & 3u)) return CBW_ERR_UNSUPPORTED;
    const int64_t count = (int64_t)desc->N * desc->C * desc->H * desc->W;
    return hip_status(launch_relu_mask_pack(desc->dtype, count, X, x_mask, 1, static_cast<hipStream_t>(stream)));
}

int cbw_nonzero_mask_pack(int32_t dtype, int64_t count, const void* t, uint32_t* bits, void* stream)
{
    if (dtype != CBW_F32 && dtype != CBW_BF16) return CBW_ERR_INVALID_ARG;
    if (count < 0 || (count > 0 && (!t || !bits))) return CBW_ERR_INVALID_ARG;
    if (count == 0) return CBW_OK;
    if (!aligned16(t) || ((uintptr_t)bits & 3u)) return CBW_ERR_UNSUPPORTED;
    return hip_status(launch_relu_mask_pack(dtype, count, t, bits, 0, static_cast<hipStream_t>(stream)));
}

int conv_bwd_data(const cbw_conv_desc* desc, const void* dY, const void* W, void* dX, void* workspace,
                  size_t workspace_bytes, void* stream)
{
    return run_bwd_data(desc, dY, W, nullptr, dX, workspace, workspace_bytes, 0, stream, false);
}

int conv_bwd_data_masked(const cbw_conv_desc* desc, const void* dY, const void* W, const uint32_t* x_mask,
                         void* dX, void* workspace, size_t workspace_bytes, uint32_t flags, void* stream)
{
    return run_bwd_data(desc, dY, W, x_mask, dX, workspace, workspace_bytes, flags, stream, true);
}

int conv_bwd_data_masked_noalloc(const cbw_conv_desc* desc, const void* dY, const void* W, const uint32_t* x_mask,
                                 void* dX, uint32_t flags, void* stream)
{
    // the same kernels as conv_bwd_data_masked on the built-in scratch, with
    // the reduction never split (no partial tiles to hold)
    DataPlan plan;
    int st = plan_data(desc, true, &plan, true);
    if (st != CBW_OK) return st;
    if (plan.total > kNoAllocScratchBytes) return CBW_ERR_WORKSPACE;
    void* ws = nullptr;
    if ((st = scratch_for_current_device(&ws)) != CBW_OK) return st;
    return run_bwd_data(desc, dY, W, x_mask, dX, ws, kNoAllocScratchBytes, flags, stream, true, true);
}

int conv_fwd_relu_mask(const cbw_conv_desc* desc, const void* X, const void* W, void* Y, uint32_t* y_mask,
                       void* workspace, size_t workspace_bytes, void* stream)
{
    return run_fwd(desc, X, W, Y, y_mask, workspace, workspace_bytes, stream);
}

// A number per weight-gradient call that skips: the occupancy pass stores it
// as the call's dead-block flag, the GEMM compares it (a flag left by an
// earlier call, or uninitialised memory, can only send a call down the
// ranking path, which is always correct).
static uint32_t next_call_number()
{
    static std::atomic<uint32_t> counter{0};
    uint32_t g;
    do g = counter.fetch_add(1, std::memory_order_relaxed) + 1; while (g == 0);
    return g;
}

// Occupancy pass of the weight gradient on NHWC tensors (dY, and the
// footprints, in NHWC order): dY block occupancy from dy_mask or dY, and
// with x_skip the X-window liveness from the packed X footprint xbits.
static OccParams weight_occ_params(const cbw_conv_desc* desc, const WeightPlan& plan, const void* dY,
                                   const uint32_t* dy_mask, bool x_skip, const uint32_t* xbits, void* workspace,
                                   uint32_t gen)
{
    OccParams op{};
    op.any_dead = at<int>(workspace, plan.header) + kDeadWord;
    op.gen = gen;
    op.dy = dY;
    op.bits = dy_mask;
    op.occ = at<uint8_t>(workspace, plan.occ);
    op.npq = (int)plan.npq;
    op.K = desc->K;
    op.chunk = plan.chunk;
    op.BNk = plan.bk;
    op.ktiles = plan.ktiles;
    op.nchunks = plan.nchunks;
    op.div_chunk = make_fastdiv((uint32_t)plan.chunk);
    op.div_ktiles = make_fastdiv((uint32_t)plan.ktiles);
    // chunks per workgroup: enough workgroups for two per CU, at most about
    // eight (pixel, k tile) pairs per thread (one with X-window liveness,
    // whose test loops over taps), within the per-chunk flag arrays (1024
    // entries each)
    const int ncombo = x_skip ? plan.tgroups * plan.ctiles : 1;
    const int per_chunk = plan.chunk * plan.ktiles;
    const int spread = (plan.nchunks + 2 * CBW_NUM_CUS - 1) / (2 * CBW_NUM_CUS);
    op.cpw = std::max(1, std::min(std::min((x_skip ? 256 : 2048) / per_chunk, spread),
                                  1024 / std::max(plan.ktiles, ncombo)));
    op.dtype = desc->dtype;
    if (x_skip) {
        op.xbits = xbits;
        op.xlive = at<uint8_t>(workspace, plan.xlive);
        op.N = desc->N; op.H = desc->H; op.W = desc->W; op.C = desc->C; op.P = desc->P; op.Q = desc->Q;
        op.S = desc->S; op.RS = desc->R * desc->S;
        op.stride_h = desc->stride_h; op.stride_w = desc->stride_w;
        op.pad_h = desc->pad_h; op.pad_w = desc->pad_w;
        op.tpg = plan.tpg;
        op.tgroups = plan.tgroups;
        op.ctiles = plan.ctiles;
        op.ctw = plan.tpg > 1 ? desc->C : weight_tile_channels();
        op.div_q = make_fastdiv((uint32_t)desc->Q);
        op.div_p = make_fastdiv((uint32_t)desc->P);
    }
    return op;
}

// Kernel parameters of the weight-gradient GEMM on NHWC X and dY.
static WeightParams weight_gemm_params(const cbw_conv_desc* desc, const WeightPlan& plan, const void* X,
                                       const void* dY, float* dW, void* workspace, bool skip, bool x_skip,
                                       uint32_t flags)
{
    WeightParams p{};
    p.x = X;
    p.dy = dY;
    p.out = plan.direct ? dW : at<float>(workspace, plan.partials);
    p.occ = skip ? at<uint8_t>(workspace, plan.occ) : nullptr;
    p.xlive = skip && x_skip ? at<uint8_t>(workspace, plan.xlive) : nullptr;
    p.work_slots = at<int32_t>(workspace, plan.work_slots);
    p.skip_slots = at<int32_t>(workspace, plan.skip_slots);
    p.header = at<int>(workspace, plan.header);
    p.N = desc->N; p.H = desc->H; p.W = desc->W; p.C = desc->C; p.K = desc->K; p.R = desc->R; p.S = desc->S;
    p.P = desc->P; p.Q = desc->Q;
    p.stride_h = desc->stride_h; p.stride_w = desc->stride_w; p.pad_h = desc->pad_h; p.pad_w = desc->pad_w;
    p.npq = (int)plan.npq;
    p.nchunks = plan.nchunks;
    p.chunks_per_split = plan.chunks_per_split;
    p.ctiles = plan.ctiles;
    p.ktiles = plan.ktiles;
    p.nsplit = plan.nsplit;
    p.bk = plan.bk;
    p.tpg = plan.tpg;
    p.tgroups = plan.tgroups;
    p.cg = plan.cg;
    p.rows = plan.rows ? 1 : 0;
    p.mode_flags = (int)flags;
    p.div_q = make_fastdiv((uint32_t)desc->Q);
    p.div_p = make_fastdiv((uint32_t)desc->P);
    p.x_bytes = (uint32_t)((int64_t)desc->N * desc->H * desc->W * desc->C * elem_bytes(desc->dtype));
    p.dy_bytes = (uint32_t)(plan.npq * desc->K * elem_bytes(desc->dtype));
    return p;
}

// Weight gradient; x_skip also skips blocks whose X operand is all zero.
static int run_weight(const cbw_conv_desc* desc, const void* X, const void* dY, const uint32_t* x_mask,
               const uint32_t* dy_mask, bool x_skip, float* dW, void* workspace, size_t workspace_bytes,
               uint32_t flags, void* stream)
{
    WeightPlan plan;
    int st = plan_weight(desc, &plan, !x_skip);   // X-block skipping runs the chunked kernel
    if (st != CBW_OK) return st;
    if (!X || !dY || !dW) return CBW_ERR_INVALID_ARG;
    if (!aligned16(X) || !aligned16(dY) || !aligned16(dW) || !aligned16(dy_mask) || !aligned16(x_mask))
        return CBW_ERR_UNSUPPORTED;
    if ((st = check_ws(workspace, workspace_bytes, plan.total)) != CBW_OK) return st;
    if (!tiles_consistent()) return CBW_ERR_UNSUPPORTED;
    if (x_skip && plan.tgroups * plan.ctiles > 1024) return CBW_ERR_UNSUPPORTED;   // liveness flags per chunk
    const uint32_t gen = next_call_number();
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool skip = !(flags & CBW_FLAG_NO_SKIP);
    hipError_t e;
    if (desc->act_layout == CBW_NCHW) {
        // the kernels read NHWC copies of X and dY (and NHWC-order footprints)
        void* tx = at<void>(workspace, plan.t_x);
        void* tdy = at<void>(workspace, plan.t_dy);
        if ((e = launch_transpose(desc->dtype, X, tx, desc->N, desc->C, desc->H * desc->W, s)) != hipSuccess ||
            (e = launch_transpose(desc->dtype, dY, tdy, desc->N, desc->K, desc->P * desc->Q, s)) != hipSuccess)
            return hip_status(e);
        X = tx;
        dY = tdy;
        if (skip && dy_mask) {
            uint32_t* t = at<uint32_t>(workspace, plan.t_dymask);
            if ((e = launch_bits_nchw_to_nhwc(dy_mask, t, desc->N, desc->K, desc->P * desc->Q, s)) != hipSuccess)
                return hip_status(e);
            dy_mask = t;
        }
        if (skip && x_skip && x_mask) {
            uint32_t* t = at<uint32_t>(workspace, plan.xbits);
            if ((e = launch_bits_nchw_to_nhwc(x_mask, t, desc->N, desc->C, desc->H * desc->W, s)) != hipSuccess)
                return hip_status(e);
            x_mask = t;
        }
    }
    if (skip) {
        const uint32_t* xbits = x_mask;
        if (x_skip && !xbits) {
            // the X-window liveness is read from a packed footprint of X: the
            // caller's, or one packed here from X's non-zeros
            uint32_t* packed = at<uint32_t>(workspace, plan.xbits);
            const int64_t count = (int64_t)desc->N * desc->H * desc->W * desc->C;
            if ((e = launch_relu_mask_pack(desc->dtype, count, X, packed, 0, s)) != hipSuccess)
                return hip_status(e);
            xbits = packed;
        }
        const OccParams op = weight_occ_params(desc, plan, dY, dy_mask, x_skip, xbits, workspace, gen);
        if ((e = launch_occupancy(op, s)) != hipSuccess) return hip_status(e);
    }
    WeightParams p = weight_gemm_params(desc, plan, X, dY, dW, workspace, skip, x_skip, flags);
    p.gen = gen;
    if ((e = launch_bwd_weight(desc->dtype, p, s, prof_events(1))) != hipSuccess) return hip_status(e);
    if (!plan.direct) {
        e = launch_splitk_reduce(p.out, dW, plan.nparts, desc->K, desc->R * desc->S, desc->C,
                                 desc->w_layout == CBW_KRSC, s);
        if (e != hipSuccess) return hip_status(e);
    }
    return CBW_OK;
}

// Both gradients of one layer.  NHWC: one preparation launch (filter
// transform, compaction counts, dY occupancy), then with the tiled data
// gradient the weight GEMM, the data GEMM (the weight gradient's split-K
// reduction in its tail workgroups) and, when the data gradient may split,
// its split reduction; with the row-window or pointwise data gradient the
// data GEMM, the weight GEMM and one reduction launch.  NCHW: the two
// separate calls on the two parts of the workspace.
static int run_bwd_both(const cbw_conv_desc* desc, const void* X, const void* dY, const void* W,
                        const uint32_t* x_mask, const uint32_t* dy_mask, void* dX, float* dW, void* ws,
                        size_t ws_bytes, uint32_t flags, void* stream)
{
    if (flags & ~(CBW_FLAG_NO_SKIP | CBW_FLAG_SKIP_X_BLOCKS)) return CBW_ERR_INVALID_ARG;
    size_t off = 0, total = 0;
    int st = both_offset(desc, &off, &total);
    if (st != CBW_OK) return st;
    const bool masked = x_mask != nullptr;
    const bool skip = !(flags & CBW_FLAG_NO_SKIP);
    const bool x_skip = skip && masked && (flags & CBW_FLAG_SKIP_X_BLOCKS);
    DataPlan dplan;
    WeightPlan wplan;
    if ((st = plan_data(desc, masked, &dplan)) != CBW_OK) return st;
    if ((st = plan_weight(desc, &wplan, !x_skip)) != CBW_OK) return st;
    const bool want_dx = dX != nullptr;   // NULL: the weight gradient alone (a first layer's input has no gradient)
    if (!X || !dY || !dW || (want_dx && !W)) return CBW_ERR_INVALID_ARG;
    if (!aligned16(X) || !aligned16(dY) || !aligned16(W) || !aligned16(dX) || !aligned16(dW) ||
        !aligned16(x_mask) || !aligned16(dy_mask))
        return CBW_ERR_UNSUPPORTED;
    if ((st = check_ws(ws, ws_bytes, total)) != CBW_OK) return st;
    if (!tiles_consistent()) return CBW_ERR_UNSUPPORTED;
    if (x_skip && wplan.tgroups * wplan.ctiles > 1024) return CBW_ERR_UNSUPPORTED;   // liveness flags per chunk
    void* wws = static_cast<char*>(ws) + off;
    if (!want_dx)
        return run_weight(desc, X, dY, x_skip ? x_mask : nullptr, dy_mask, x_skip, dW, wws, total - off,
                          flags & CBW_FLAG_NO_SKIP, stream);
    if (desc->act_layout == CBW_NCHW) {
        st = run_bwd_data(desc, dY, W, x_mask, dX, ws, off, flags & CBW_FLAG_NO_SKIP, stream, masked);
        if (st != CBW_OK) return st;
        return run_weight(desc, X, dY, x_skip ? x_mask : nullptr, dy_mask, x_skip, dW, wws, total - off,
                          flags & CBW_FLAG_NO_SKIP, stream);
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool tiled = !dplan.rows && !dplan.pw;   // the tiled GEMM (else a dedicated kernel)
    const bool gather = tiled && data_gathers(dplan, masked, flags);
    const int mode = dplan.rows ? MODE_ROWS
                     : dplan.pw ? MODE_PW
                                : (!masked ? MODE_DENSE : (gather ? MODE_GATHER : MODE_SELECT));
    int* header = at<int>(ws, dplan.header);
    void* wt = at<void>(ws, dplan.wt);
    DataParams dp{};
    CompactParams cp;
    if (tiled) data_gemm_params(desc, dplan, dY, wt, x_mask, dX, ws, gather, false, &dp, &cp);
    OccParams op{};
    const uint32_t gen = next_call_number();
    if (skip) op = weight_occ_params(desc, wplan, dY, dy_mask, x_skip, x_mask, wws, gen);
    hipError_t e = launch_data_prep(desc->dtype, W, wt, desc->K, desc->C, desc->R * desc->S,
                                    desc->w_layout == CBW_KRSC, header, mode, gather ? &cp : nullptr, s,
                                    skip ? &op : nullptr);
    if (e != hipSuccess) return hip_status(e);
    WeightParams wp = weight_gemm_params(desc, wplan, X, dY, dW, wws, skip, x_skip, flags & CBW_FLAG_NO_SKIP);
    wp.gen = gen;
    ReduceParams rp{};
    if (!wplan.direct) {
        const int64_t n4 = (int64_t)desc->K * desc->R * desc->S * desc->C / 4;
        rp.part = wp.out;
        rp.dw = dW;
        rp.nsplit = wplan.nparts;
        rp.K = desc->K;
        rp.RS = desc->R * desc->S;
        rp.C = desc->C;
        rp.krsc = desc->w_layout == CBW_KRSC;
        rp.G = splitk_reduce_group(wplan.nparts, n4);
        rp.blocks = (int)((n4 * rp.G + 255) / 256);
    }
    if (tiled) {
        // The weight gradient first; its split-K reduction then runs in
        // tail workgroups of the data-gradient GEMM launch, on the CUs that
        // the GEMM's last round of tiles leaves idle, and only the data
        // gradient's own split reduction (gather mode, or a split dense
        // tiling) keeps a launch of its own.
        if ((e = launch_bwd_weight(desc->dtype, wp, s, prof_events(1))) != hipSuccess) return hip_status(e);
        dp.dw_red = rp;
        if ((e = launch_bwd_data(desc->dtype, mode, dp, s, prof_events(0), false)) != hipSuccess) return hip_status(e);
        const bool dx_reduce = mode == MODE_GATHER || dplan.split > 1;
        if (!dx_reduce) return CBW_OK;
        return hip_status(launch_bwd_reduce(desc->dtype, mode, dp, true, ReduceParams{}, s));
    }
    if (dplan.rows) {
        const DataRowsParams rwp = data_rows_params(desc, dplan, dY, wt, x_mask, dX, ws, skip);
        e = launch_bwd_data_rows(rwp, dplan.rows_grid, dplan.rows_nbw, s, prof_events(0));
    } else {
        const DataPwParams pp = data_pw_params(desc, dplan, dY, wt, x_mask, dX, ws, skip);
        e = launch_bwd_data_pw(pp, dplan.pw_grid, s, prof_events(0));
    }
    if (e != hipSuccess) return hip_status(e);
    if ((e = launch_bwd_weight(desc->dtype, wp, s, prof_events(1))) != hipSuccess) return hip_status(e);
    return hip_status(launch_bwd_reduce(desc->dtype, mode, dp, false, rp, s));
}

int conv_bwd_data_elementwise(const cbw_conv_desc* desc, const void* dY, const void* W, const uint32_t* x_mask,
                              void* dX, void* workspace, size_t workspace_bytes, void* stream)
{
    int st = validate_elementwise(desc);
    if (st != CBW_OK) return st;
    if (!dY || !W || !dX || !x_mask) return CBW_ERR_INVALID_ARG;
    if (!aligned16(dY) || !aligned16(W) || !aligned16(dX) || !aligned16(x_mask)) return CBW_ERR_UNSUPPORTED;
    if ((st = check_ws(workspace, workspace_bytes, elementwise_ws(desc))) != CBW_OK) return st;
    EwParams p{};
    p.dy = dY;
    p.w = W;
    p.mask = x_mask;
    p.dx = dX;
    p.counts = static_cast<int32_t*>(workspace);
    p.N = desc->N; p.H = desc->H; p.W = desc->W; p.C = desc->C; p.K = desc->K; p.R = desc->R; p.S = desc->S;
    p.P = desc->P; p.Q = desc->Q;
    p.stride_h = desc->stride_h; p.stride_w = desc->stride_w; p.pad_h = desc->pad_h; p.pad_w = desc->pad_w;
    p.npix = desc->N * desc->H * desc->W;
    p.dy_bytes = (uint32_t)((int64_t)desc->N * desc->P * desc->Q * desc->K * 2);
    p.w_bytes = (uint32_t)((int64_t)desc->K * desc->R * desc->S * desc->C * 2);
    p.dx_bytes = (uint32_t)((int64_t)p.npix * desc->C * 2);
    p.div_w = make_fastdiv((uint32_t)desc->W);
    p.div_h = make_fastdiv((uint32_t)desc->H);
    return hip_status(launch_elementwise_data(p, static_cast<hipStream_t>(stream)));
}

int cbw_read_pixel_counts(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes,
                          int32_t* counts, int64_t* total, void* stream)
{
    int st = validate_elementwise(desc);
    if (st != CBW_OK) return st;
    if (!workspace || !total) return CBW_ERR_INVALID_ARG;
    if (workspace_bytes < elementwise_ws(desc)) return CBW_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t npix = (int64_t)desc->N * desc->H * desc->W;
    const int32_t* src = static_cast<const int32_t*>(workspace);
    int64_t sum = 0;
    int32_t buf[4096];
    for (int64_t i0 = 0; i0 < npix; i0 += 4096) {
        const int64_t n = npix - i0 < 4096 ? npix - i0 : 4096;
        hipError_t e = hipMemcpyAsync(buf, src + i0, n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_status(e);
        for (int64_t i = 0; i < n; ++i) sum += buf[i];
        if (counts) std::memcpy(counts + i0, buf, n * sizeof(int32_t));
    }
    *total = sum;
    return CBW_OK;
}

int conv_bwd_weight_sparse(const cbw_conv_desc* desc, const void* X, const void* dY, const uint32_t* dy_mask,
                           float* dW, void* workspace, size_t workspace_bytes, uint32_t flags, void* stream)
{
    return run_weight(desc, X, dY, nullptr, dy_mask, false, dW, workspace, workspace_bytes, flags, stream);
}

int conv_bwd_weight_sparse_x(const cbw_conv_desc* desc, const void* X, const void* dY, const uint32_t* x_mask,
                             const uint32_t* dy_mask, float* dW, void* workspace, size_t workspace_bytes,
                             uint32_t flags, void* stream)
{
    return run_weight(desc, X, dY, x_mask, dy_mask, true, dW, workspace, workspace_bytes, flags, stream);
}

int conv_bwd_sparse(const cbw_conv_desc* desc, const void* X, const void* dY, const void* W, const uint32_t* x_mask,
                    const uint32_t* dy_mask, void* dX, float* dW, void* workspace, size_t workspace_bytes,
                    uint32_t flags, void* stream)
{
    return run_bwd_both(desc, X, dY, W, x_mask, dy_mask, dX, dW, workspace, workspace_bytes, flags, stream);
}

int cbw_read_weight_work(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, int32_t* work,
                         int32_t* nsplit, int32_t* ntiles, void* stream)
{
    WeightPlan plan;
    if (!workspace || !nsplit || !ntiles) return CBW_ERR_INVALID_ARG;
    int st = last_weight_plan(desc, workspace, workspace_bytes, &plan, static_cast<hipStream_t>(stream));
    if (st != CBW_OK) return st;
    *nsplit = plan.nsplit;
    *ntiles = plan.grid / plan.nsplit;
    if (!work) return CBW_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(work, at<int32_t>(const_cast<void*>(workspace), plan.work_slots),
                                  (size_t)plan.grid * sizeof(int32_t), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    return hip_status(e);
}

int cbw_read_stats(const cbw_conv_desc* desc, int op, const void* workspace, size_t workspace_bytes,
                   cbw_stats* out, void* stream)
{
    if (!out || !workspace) return CBW_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    cbw_stats r{};
    int st;
    if (op == CBW_OP_BWD_BOTH) {
        // data-gradient rows from the first part, weight-gradient blocks from the second
        size_t off, total;
        if ((st = both_offset(desc, &off, &total)) != CBW_OK) return st;
        if (workspace_bytes < total) return CBW_ERR_WORKSPACE;
        cbw_stats d{}, w{};
        if ((st = cbw_read_stats(desc, CBW_OP_BWD_DATA_MASKED, workspace, off, &d, stream)) != CBW_OK) return st;
        if ((st = cbw_read_stats(desc, CBW_OP_BWD_WEIGHT, static_cast<const char*>(workspace) + off, total - off, &w,
                                 stream)) != CBW_OK)
            return st;
        r.rows_total = d.rows_total;
        r.rows_live = d.rows_live;
        r.blocks_total = w.blocks_total;
        r.blocks_skipped = w.blocks_skipped;
        *out = r;
        return CBW_OK;
    }
    if (op == CBW_OP_BWD_DATA || op == CBW_OP_BWD_DATA_MASKED) {
        DataPlan plan;
        if ((st = plan_data(desc, op == CBW_OP_BWD_DATA_MASKED, &plan)) != CBW_OK) return st;
        if (workspace_bytes < plan.total) return CBW_ERR_WORKSPACE;
        int header = 0;
        hipError_t e = hipMemcpyAsync(&header, at<void>(const_cast<void*>(workspace), plan.header), sizeof(int),
                                      hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_status(e);
        r.rows_total = (int64_t)plan.groups * plan.npix;
        r.rows_live = r.rows_total;
        if (plan.rows && header == MODE_ROWS) {
            // pixels of the rows each workgroup computed (dead rows skipped)
            int32_t buf[256];
            int64_t live = 0;
            const int32_t* slots = at<int32_t>(const_cast<void*>(workspace), plan.row_counts);
            for (int i0 = 0; i0 < plan.rows_grid; i0 += 256) {
                const int n = plan.rows_grid - i0 < 256 ? plan.rows_grid - i0 : 256;
                e = hipMemcpyAsync(buf, slots + i0, n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
                if (e == hipSuccess) e = hipStreamSynchronize(s);
                if (e != hipSuccess) return hip_status(e);
                for (int i = 0; i < n; ++i) live += buf[i];
            }
            r.rows_live = live / 2 * plan.groups;   // each pixel is counted by its two channel-half waves
        } else if (plan.pw && header == MODE_PW) {
            // pixels of the 16-pixel blocks each workgroup computed (dead blocks skipped)
            int32_t buf[256];
            int64_t live = 0;
            const int32_t* slots = at<int32_t>(const_cast<void*>(workspace), plan.row_counts);
            for (int i0 = 0; i0 < plan.pw_grid; i0 += 256) {
                const int n = plan.pw_grid - i0 < 256 ? plan.pw_grid - i0 : 256;
                e = hipMemcpyAsync(buf, slots + i0, n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
                if (e == hipSuccess) e = hipStreamSynchronize(s);
                if (e != hipSuccess) return hip_status(e);
                for (int i = 0; i < n; ++i) live += buf[i];
            }
            r.rows_live = live * plan.groups;
        } else if (op == CBW_OP_BWD_DATA_MASKED && header == MODE_GATHER) {
            int32_t counts[64];
            int64_t live = 0;
            for (int g0 = 0; g0 < plan.groups; g0 += 64) {
                const int n = plan.groups - g0 < 64 ? plan.groups - g0 : 64;
                e = hipMemcpyAsync(counts, at<int32_t>(const_cast<void*>(workspace), plan.counts) + g0,
                                   n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
                if (e == hipSuccess) e = hipStreamSynchronize(s);
                if (e != hipSuccess) return hip_status(e);
                for (int i = 0; i < n; ++i) live += counts[i];
            }
            r.rows_live = live;
        }
    } else if (op == CBW_OP_BWD_WEIGHT) {
        WeightPlan plan;
        if ((st = last_weight_plan(desc, workspace, workspace_bytes, &plan, s)) != CBW_OK) return st;
        r.blocks_total = (int64_t)plan.nchunks * plan.ktiles * plan.tgroups * plan.ctiles;
        int64_t skipped = 0;
        int32_t buf[256];
        const int32_t* slots = at<int32_t>(const_cast<void*>(workspace), plan.skip_slots);
        for (int i0 = 0; i0 < plan.grid; i0 += 256) {
            const int n = plan.grid - i0 < 256 ? plan.grid - i0 : 256;
            hipError_t e = hipMemcpyAsync(buf, slots + i0, n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
            if (e == hipSuccess) e = hipStreamSynchronize(s);
            if (e != hipSuccess) return hip_status(e);
            for (int i = 0; i < n; ++i) skipped += buf[i];
        }
        r.blocks_skipped = skipped;
    } else {
        return CBW_ERR_INVALID_ARG;
    }
    *out = r;
    return CBW_OK;
}

int cbw_set_profile_events(int op, void* start, void* stop)
{
    int fam;
    if (op == CBW_OP_BWD_DATA || op == CBW_OP_BWD_DATA_MASKED) fam = 0;
    else if (op == CBW_OP_BWD_WEIGHT) fam = 1;
    else if (op == CBW_OP_FWD) fam = 2;
    else return CBW_ERR_INVALID_ARG;
    if ((start == nullptr) != (stop == nullptr)) return CBW_ERR_INVALID_ARG;
    g_prof[fam][0] = static_cast<hipEvent_t>(start);
    g_prof[fam][1] = static_cast<hipEvent_t>(stop);
    return CBW_OK;
}

int cbw_read_live_lists(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, int group,
                        int32_t* pixels, int32_t* count, int32_t* group_width, void* stream)
{
    DataPlan plan;
    int st = plan_data(desc, true, &plan);
    if (st != CBW_OK) return st;
    if (!workspace || !count || !group_width || group < 0 || group >= plan.groups) return CBW_ERR_INVALID_ARG;
    if (workspace_bytes < plan.total) return CBW_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* ws = const_cast<void*>(workspace);
    if (plan.rows || plan.pw) return CBW_ERR_UNSUPPORTED;   // the row-window and pointwise kernels list nothing
    int32_t n = 0;
    hipError_t e = hipMemcpyAsync(&n, at<int32_t>(ws, plan.counts) + group, sizeof(int32_t),
                                  hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_status(e);
    if (n < 0 || n > plan.npix) return CBW_ERR_INVALID_ARG;  // workspace not written by a gather call
    *count = n;
    *group_width = plan.bm;
    if (pixels && n == plan.npix) {
        // a fully live group's list (0, 1, 2, ...) is never stored
        for (int32_t i = 0; i < n; ++i) pixels[i] = i;
    } else if (pixels && n > 0) {
        e = hipMemcpyAsync(pixels, at<int32_t>(ws, plan.lists) + (int64_t)group * plan.npix,
                           (size_t)n * sizeof(int32_t), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_status(e);
    }
    return CBW_OK;
}

int cbw_read_occupancy(const cbw_conv_desc* desc, const void* workspace, size_t workspace_bytes, uint8_t* occ,
                       int32_t* nchunks, int32_t* ktiles, int32_t* chunk_pixels, int32_t* ktile_width,
                       void* stream)
{
    WeightPlan plan;
    if (!workspace || !nchunks || !ktiles || !chunk_pixels || !ktile_width) return CBW_ERR_INVALID_ARG;
    int st = last_weight_plan(desc, workspace, workspace_bytes, &plan, static_cast<hipStream_t>(stream));
    if (st != CBW_OK) return st;
    *nchunks = plan.nchunks;
    *ktiles = plan.ktiles;
    *chunk_pixels = plan.chunk;
    *ktile_width = plan.bk;
    if (occ) {
        hipStream_t s = static_cast<hipStream_t>(stream);
        hipError_t e = hipMemcpyAsync(occ, at<uint8_t>(const_cast<void*>(workspace), plan.occ),
                                      (size_t)plan.nchunks * plan.ktiles, hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return hip_status(e);
    }
    return CBW_OK;
}

}  // extern "C"
