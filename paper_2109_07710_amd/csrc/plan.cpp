// Host-only validation and workspace planning (see plan.hpp).
#include "plan.hpp"

namespace cbw {

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

Region take(size_t* cursor, size_t bytes)
{
    Region r;
    r.off = *cursor;
    r.bytes = bytes;
    *cursor = align256(*cursor + bytes);
    return r;
}

constexpr int64_t kMaxElems = (int64_t)1 << 31;

}  // namespace

int validate_desc(const cbw_conv_desc* d)
{
    if (!d) return CBW_ERR_INVALID_ARG;
    if (d->N <= 0 || d->C <= 0 || d->H <= 0 || d->W <= 0 || d->K <= 0 || d->R <= 0 || d->S <= 0)
        return CBW_ERR_INVALID_ARG;
    if (d->stride_h <= 0 || d->stride_w <= 0 || d->pad_h < 0 || d->pad_w < 0) return CBW_ERR_INVALID_ARG;
    const int64_t ph = (int64_t)d->H + 2 * (int64_t)d->pad_h - d->R;
    const int64_t pw = (int64_t)d->W + 2 * (int64_t)d->pad_w - d->S;
    if (ph < 0 || pw < 0) return CBW_ERR_INVALID_ARG;
    if (d->P != ph / d->stride_h + 1 || d->Q != pw / d->stride_w + 1) return CBW_ERR_INVALID_ARG;
    if (d->dtype != CBW_F32 && d->dtype != CBW_BF16) return CBW_ERR_INVALID_ARG;
    if (d->act_layout != CBW_NHWC && d->act_layout != CBW_NCHW) return CBW_ERR_INVALID_ARG;
    if (d->w_layout != CBW_KRSC && d->w_layout != CBW_KCRS) return CBW_ERR_INVALID_ARG;
    const int E = d->dtype == CBW_BF16 ? 8 : 4;
    if (d->C % E != 0 || d->K % E != 0) return CBW_ERR_UNSUPPORTED;
    const int64_t npix = (int64_t)d->N * d->H * d->W, npq = (int64_t)d->N * d->P * d->Q;
    if (npix * d->C >= kMaxElems || npq * d->K >= kMaxElems) return CBW_ERR_UNSUPPORTED;
    // every tensor the kernels read through a buffer descriptor stays below 2^31 bytes
    const int64_t esz = d->dtype == CBW_BF16 ? 2 : 4;
    if (npix * d->C * esz >= kMaxElems || npq * d->K * esz >= kMaxElems) return CBW_ERR_UNSUPPORTED;
    // the fp32 weight gradient (and each split partial of it) stays below 2^31 bytes
    if ((int64_t)d->K * d->C * d->R * d->S * 4 >= kMaxElems) return CBW_ERR_UNSUPPORTED;
    if (d->K > 1024 * kWeightTileK) return CBW_ERR_UNSUPPORTED;  // occupancy flags per chunk
    return CBW_OK;
}

int require_nhwc(const cbw_conv_desc* d)
{
    const int st = validate_desc(d);
    if (st != CBW_OK) return st;
    return d->act_layout == CBW_NHWC ? CBW_OK : CBW_ERR_UNSUPPORTED;
}

int data_tile_index(int C)
{
    int best = 0, best_waste = -1;
    for (int t = 0; t < kDataTileCount; ++t) {
        const int bm = kDataTiles[t].bm;
        const int waste = (C + bm - 1) / bm * bm - C;
        if (8 * waste <= C) return t;
        if (best_waste < 0 || waste < best_waste) {
            best = t;
            best_waste = waste;
        }
    }
    return best;
}

bool data_rows_eligible(const cbw_conv_desc* d)
{
    return d->dtype == CBW_BF16 && d->R == 3 && d->S == 3 && d->stride_h == 1 && d->stride_w == 1 && d->C == 64 &&
           d->K == 64;
}

bool data_pw_eligible(const cbw_conv_desc* d)
{
    auto ok = [](int c) { return c == 64 || c == 128 || c == 256; };
    return d->dtype == CBW_BF16 && d->R == 1 && d->S == 1 && d->stride_h == 1 && d->stride_w == 1 &&
           d->pad_h == 0 && d->pad_w == 0 && ok(d->C) && ok(d->K) && d->C * d->K <= 16384;
}

int plan_data(const cbw_conv_desc* d, bool masked, DataPlan* out, bool no_split, bool allow_rows)
{
    int st = validate_desc(d);
    if (st != CBW_OK) return st;
    DataPlan p;
    if (allow_rows && data_pw_eligible(d)) {
        // as many resident waves as give every wave the same whole number of
        // 16-pixel blocks (the last wave takes the rest)
        p.tile = data_tile_index(d->C);
        p.bm = kDataTiles[p.tile].bm;
        p.bn = kDataTiles[p.tile].bn;
        p.npix = (int64_t)d->N * d->H * d->W;
        p.groups = (d->C + p.bm - 1) / p.bm;
        p.pw = true;
        const int64_t nblk = (p.npix + 15) / 16;
        p.pw_bpw = (int)((nblk + kDataPwMaxWaves - 1) / kDataPwMaxWaves);
        const int64_t waves = (nblk + p.pw_bpw - 1) / p.pw_bpw;
        p.pw_grid = (int)((waves + kDataPwWaves - 1) / kDataPwWaves);
        size_t cur = 0;
        p.header = take(&cur, 256);
        p.wt = take(&cur, (size_t)d->K * d->C * elem_bytes(d->dtype));
        p.row_counts = take(&cur, (size_t)p.pw_grid * 4);
        if (d->act_layout == CBW_NCHW) {
            p.t_dy = take(&cur, (size_t)d->N * d->P * d->Q * d->K * elem_bytes(d->dtype));
            p.t_dx = take(&cur, (size_t)p.npix * d->C * elem_bytes(d->dtype));
            if (masked) p.t_mask = take(&cur, ((size_t)p.npix * d->C + 31) / 32 * 4);
        }
        p.total = cur;
        *out = p;
        return CBW_OK;
    }
    if (allow_rows && data_rows_eligible(d)) {
        // one workgroup per CU: strips of consecutive output rows, as many
        // as make the segments times the strips fill the CUs once
        p.tile = data_tile_index(d->C);
        p.bm = kDataTiles[p.tile].bm;
        p.bn = kDataTiles[p.tile].bn;
        p.npix = (int64_t)d->N * d->H * d->W;
        p.groups = (d->C + p.bm - 1) / p.bm;
        p.rows = true;
        p.rows_nseg = (d->W + kDataRowsSegment - 1) / kDataRowsSegment;
        const int nrows = d->N * d->H;
        int strips = CBW_NUM_CUS / p.rows_nseg;
        if (strips < 1) strips = 1;
        p.rows_per_strip = (nrows + strips - 1) / strips;
        p.rows_grid = (nrows + p.rows_per_strip - 1) / p.rows_per_strip * p.rows_nseg;
        const int wseg = d->W < kDataRowsSegment ? d->W : kDataRowsSegment;
        p.rows_nbw = ((wseg + 15) / 16 + 3) / 4;
        // the deepest prefetch (at most 8 steps) whose rings fit the LDS:
        // depth + 3 dY rows and depth + 2 footprint rows
        // a slot holds the 16-column blocks' rows and the two halo columns
        p.rows_slot = ((wseg + 15) / 16 * 16 + 2 + 7) / 8 * 1024;
        p.rows_mslot = (wseg * 8 + 1023) / 1024 * 1024;   // whole 1 KB copies of 16-byte pieces
        p.rows_depth = 8;
        while (p.rows_depth > 1 &&
               (p.rows_depth + 3) * p.rows_slot + (p.rows_depth + 2) * p.rows_mslot > kDataRowsLds)
            --p.rows_depth;
        size_t cur = 0;
        p.header = take(&cur, 256);
        p.wt = take(&cur, (size_t)d->K * d->C * d->R * d->S * elem_bytes(d->dtype));
        p.row_counts = take(&cur, (size_t)p.rows_grid * 4);
        if (d->act_layout == CBW_NCHW) {
            p.t_dy = take(&cur, (size_t)d->N * d->P * d->Q * d->K * elem_bytes(d->dtype));
            p.t_dx = take(&cur, (size_t)p.npix * d->C * elem_bytes(d->dtype));
            if (masked) p.t_mask = take(&cur, ((size_t)p.npix * d->C + 31) / 32 * 4);
        }
        p.total = cur;
        *out = p;
        return CBW_OK;
    }
    p.tile = data_tile_index(d->C);
    p.bm = kDataTiles[p.tile].bm;
    p.bn = kDataTiles[p.tile].bn;
    p.npix = (int64_t)d->N * d->H * d->W;
    p.groups = (d->C + p.bm - 1) / p.bm;
    p.nblk = (int)((p.npix + kCompactBlock - 1) / kCompactBlock);
    size_t cur = 0;
    int cand[kDataRowChoices];
    for (int c = 0; c < kDataRowChoices; ++c) {
        const int rows = p.bn - 16 * c;
        cand[c] = p.groups * (int)((p.npix + rows - 1) / rows);
    }
    p.brows = data_rows_pick(cand, p.bn, kDataSlots);
    p.ptiles = (int)((p.npix + p.brows - 1) / p.brows);
    const int bk = 8 * (d->dtype == CBW_BF16 ? 8 : 4);
    p.nsteps = d->R * d->S * ((d->K + bk - 1) / bk);
    p.split = no_split ? 1 : host_data_split(p.ptiles * p.groups, p.nsteps);
    p.header = take(&cur, 256);
    p.wt = take(&cur, (size_t)d->K * d->C * d->R * d->S * elem_bytes(d->dtype));
    if (masked) {
        p.blk_counts = take(&cur, (size_t)p.groups * p.nblk * 4);
        p.counts = take(&cur, (size_t)p.groups * 4);
        p.dead_flags = take(&cur, (size_t)p.groups * 4);
        p.lists = take(&cur, (size_t)p.groups * p.npix * 4);
    }
    // Split partial tiles.  Without skipping the host knows the split; with
    // compaction it is decided on the device, bounded by one partial tile
    // per resident workgroup.
    const size_t tile_bytes = (size_t)p.bn * p.bm * 4;
    if (masked && !no_split) p.partial = take(&cur, (size_t)kDataSlots * tile_bytes);
    else if (p.split > 1) p.partial = take(&cur, (size_t)p.ptiles * p.groups * p.split * tile_bytes);
    if (d->act_layout == CBW_NCHW) {
        p.t_dy = take(&cur, (size_t)d->N * d->P * d->Q * d->K * elem_bytes(d->dtype));
        p.t_dx = take(&cur, (size_t)p.npix * d->C * elem_bytes(d->dtype));
        if (masked) p.t_mask = take(&cur, ((size_t)p.npix * d->C + 31) / 32 * 4);
    }
    p.total = cur;
    *out = p;
    return CBW_OK;
}

int fwd_as_data_desc(const cbw_conv_desc* d, cbw_conv_desc* out)
{
    int st = require_nhwc(d);
    if (st != CBW_OK) return st;
    if (d->stride_h != 1 || d->stride_w != 1) return CBW_ERR_UNSUPPORTED;
    if (d->pad_h > d->R - 1 || d->pad_w > d->S - 1) return CBW_ERR_UNSUPPORTED;
    cbw_conv_desc v = *d;
    v.C = d->K; v.K = d->C;
    v.H = d->P; v.W = d->Q;
    v.P = d->H; v.Q = d->W;
    v.pad_h = d->R - 1 - d->pad_h;
    v.pad_w = d->S - 1 - d->pad_w;
    if ((st = validate_desc(&v)) != CBW_OK) return st;
    *out = v;
    return CBW_OK;
}

int weight_tile_k_for(const cbw_conv_desc* d)
{
    if (d->dtype != CBW_BF16) return kWeightTileK;   // the fp32 kernel keeps 256 x 256 tiles
    if (d->K <= 64) return 64;
    if (d->K <= 128) return 128;
    return kWeightTileK;
}

int weight_taps_per_group(const cbw_conv_desc* d)
{
    const int rs = d->R * d->S;
    if (d->dtype != CBW_BF16 || rs == 1 || 2 * d->C > kWeightTileC) return 1;
    // as few groups as the tile allows, the taps spread evenly over them
    // (9 taps of 64 channels: 3 + 3 + 3 rather than 4 + 4 + 1)
    const int t = kWeightTileC / d->C;
    const int groups = (rs + t - 1) / t;
    return (rs + groups - 1) / groups;
}

bool weight_rows_eligible(const cbw_conv_desc* d)
{
    return d->dtype == CBW_BF16 && d->stride_h == 1 && d->stride_w == 1 && d->R <= 3 && d->S <= 3 &&
           d->C % 64 == 0 && d->K % 64 == 0 && d->C <= 128 && d->K <= 128;
}

int plan_weight(const cbw_conv_desc* d, WeightPlan* out, bool allow_rows)
{
    int st = validate_desc(d);
    if (st != CBW_OK) return st;
    WeightPlan p;
    p.npq = (int64_t)d->N * d->P * d->Q;
    p.rows = allow_rows && weight_rows_eligible(d);
    if (p.rows) {
        // row-window kernel: 64 x 64 (k, c) tiles, output rows in segments
        // of up to 128 columns; the skip chunks are whole output rows
        p.chunk = d->Q;
        p.nchunks = d->N * d->P;
        p.bk = 64;
        p.tpg = 1;
        p.cg = 64;
        p.tgroups = (d->Q + kRowSegment - 1) / kRowSegment;
        p.ctiles = d->C / 64;
    } else {
        p.chunk = weight_chunk_px(d->dtype);
        p.nchunks = (int)((p.npq + p.chunk - 1) / p.chunk);
        p.bk = weight_tile_k_for(d);
        p.tpg = weight_taps_per_group(d);
        p.cg = p.tpg > 1 ? d->C : kWeightTileC;
        p.tgroups = (d->R * d->S + p.tpg - 1) / p.tpg;
        p.ctiles = p.tpg > 1 ? 1 : (d->C + kWeightTileC - 1) / kWeightTileC;
    }
    p.ktiles = (d->K + p.bk - 1) / p.bk;
    const int tiles = p.tgroups * p.ctiles * p.ktiles;
    // as many splits as fit in one round of resident workgroups
    int nsplit = kWeightSlots / tiles;
    int max_split = p.nchunks / 4;  // at least four chunks per workgroup
    if (max_split < 1) max_split = 1;
    if (nsplit > max_split) nsplit = max_split;
    if (nsplit < 1) nsplit = 1;
    p.chunks_per_split = (p.nchunks + nsplit - 1) / nsplit;
    p.nsplit = (p.nchunks + p.chunks_per_split - 1) / p.chunks_per_split;
    p.grid = tiles * p.nsplit;
    // partial weight gradients to sum: one per split (and per column segment
    // for the row-window kernel)
    p.nparts = p.rows ? p.nsplit * p.tgroups : p.nsplit;
    p.direct = (p.nparts == 1 && d->w_layout == CBW_KRSC);
    size_t cur = 0;
    p.header = take(&cur, 256);
    p.occ = take(&cur, (size_t)p.nchunks * p.ktiles);
    p.xlive = take(&cur, (size_t)p.nchunks * p.tgroups * p.ctiles);
    p.xbits = take(&cur, ((size_t)d->N * d->H * d->W * d->C + 31) / 32 * 4);
    p.skip_slots = take(&cur, (size_t)p.grid * 4);
    p.work_slots = take(&cur, (size_t)p.grid * 4);
    if (!p.direct) p.partials = take(&cur, (size_t)p.nparts * d->K * d->R * d->S * d->C * 4);
    if (d->act_layout == CBW_NCHW) {
        p.t_x = take(&cur, (size_t)d->N * d->H * d->W * d->C * elem_bytes(d->dtype));
        p.t_dy = take(&cur, (size_t)p.npq * d->K * elem_bytes(d->dtype));
        p.t_dymask = take(&cur, ((size_t)p.npq * d->K + 31) / 32 * 4);
    }
    p.total = cur;
    *out = p;
    return CBW_OK;
}

}  // namespace cbw

namespace cbw {

int weight_ws_bytes(const cbw_conv_desc* d, size_t* bytes)
{
    WeightPlan a, b;
    int st = plan_weight(d, &a, true);
    if (st != CBW_OK) return st;
    if ((st = plan_weight(d, &b, false)) != CBW_OK) return st;
    *bytes = a.total > b.total ? a.total : b.total;
    return CBW_OK;
}

}  // namespace cbw
