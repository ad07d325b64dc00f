// Host-side planning: BINPACK by first-fit decreasing and the packed-batch layout
// (Algorithm 1 up to the model call; sections 3.1 and 3.2), plus the full-batching
// layout of the paper's baseline (section 4.2).  Integer work only.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <vector>

#include "prepack.h"
#include "status.h"

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

pp_status check_lengths(const int32_t* lengths, int32_t k, int32_t* max_len, int64_t* total) {
    if (k < 0) return pp::fail(PP_ERR_INVALID_ARG, "k = %d is negative", k);
    if (k > 0 && !lengths) return pp::fail(PP_ERR_INVALID_ARG, "lengths is NULL");
    int32_t m = 0;
    int64_t sum = 0;
    for (int32_t i = 0; i < k; ++i) {
        if (lengths[i] <= 0)
            return pp::fail(PP_ERR_INVALID_ARG, "prompt %d has length %d; every prompt needs >= 1 token",
                            i, lengths[i]);
        m = std::max(m, lengths[i]);
        sum += lengths[i];
    }
    if (sum > INT32_MAX) return pp::fail(PP_ERR_INVALID_ARG, "total length %lld overflows int32", (long long)sum);
    *max_len = m;
    *total = sum;
    return PP_OK;
}

pp_status check_plan_buffers(const pp_plan* p, int32_t k, int32_t C) {
    if (!p) return pp::fail(PP_ERR_INVALID_ARG, "plan is NULL");
    if (!p->row_seg_ptr || !p->seg_prompt || !p->seg_start || !p->seg_len || !p->prompt_kv_off ||
        !p->slot_seg || !p->slot_pos || !p->slot_kv || !p->qtile_seg || !p->qtile_q0 || !p->mtile_m0)
        return pp::fail(PP_ERR_INVALID_ARG, "a plan array pointer is NULL");
    int64_t need_slots = 0, need_q = 0, need_m = 0;
    pp_plan_bounds(k, C, &need_slots, &need_q, &need_m);
    if (p->slot_cap < need_slots)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL, "slot_cap %lld < %lld (k * C)", (long long)p->slot_cap,
                        (long long)need_slots);
    if (p->qtile_cap < need_q)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL, "qtile_cap %lld < %lld (k * ceil(C / %d))",
                        (long long)p->qtile_cap, (long long)need_q, PP_QTILE);
    if (p->mtile_cap < need_m)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL, "mtile_cap %lld < %lld (ceil(k * C / %d))",
                        (long long)p->mtile_cap, (long long)need_m, PP_MTILE);
    return PP_OK;
}

// Row tiles of the projection GEMMs: the first slot of every PP_MTILE-slot tile of the batch
// that holds a slot of some span, ascending.  Tiles of row-tail padding alone are left out, so
// the GEMMs schedule (and balance across the chip) only tiles that have work.
void build_mtiles(pp_plan* p, int64_t T) {
    int32_t n = 0;
    for (int64_t t0 = 0; t0 < T; t0 += PP_MTILE) {
        const int64_t t1 = std::min<int64_t>(t0 + PP_MTILE, T);
        for (int64_t t = t0; t < t1; ++t)
            if (p->slot_seg[t] >= 0) {
                p->mtile_m0[n++] = static_cast<int32_t>(t0);
                break;
            }
    }
    p->n_mtiles = n;
}

// Attention work list: one entry per (segment, query tile).  The tiles of a segment are
// consecutive, segments longest first (ties by segment index), and inside a segment the tiles
// with more keys to visit come first (the last query tile first).  The set is fixed by the
// segments; the order serves the kernel: the tiles of one prompt, which all read the same
// keys and values, run at the same time on the same XCD (its L2 serves the re-reads), and
// long work starts first.
void build_qtiles(pp_plan* p, int32_t n_seg) {
    struct T { int32_t work, seg, q0; };
    std::vector<T> tiles;
    for (int32_t s = 0; s < n_seg; ++s)
        for (int32_t q0 = 0; q0 < p->seg_len[s]; q0 += PP_QTILE)
            tiles.push_back({std::min(q0 + PP_QTILE, p->seg_len[s]), s, q0});
    const int32_t* len = p->seg_len;
    std::stable_sort(tiles.begin(), tiles.end(), [len](const T& a, const T& b) {
        if (len[a.seg] != len[b.seg]) return len[a.seg] > len[b.seg];
        if (a.seg != b.seg) return a.seg < b.seg;
        return a.work > b.work;
    });
    for (size_t i = 0; i < tiles.size(); ++i) {
        p->qtile_seg[i] = tiles[i].seg;
        p->qtile_q0[i] = tiles[i].q0;
    }
    p->n_qtiles = static_cast<int32_t>(tiles.size());
}

void prefix_offsets(const int32_t* lengths, int32_t k, int32_t* off) {
    off[0] = 0;
    for (int32_t i = 0; i < k; ++i) off[i + 1] = off[i] + lengths[i];
}

}  // namespace

extern "C" pp_status pp_plan_bounds(int32_t k, int32_t C, int64_t* slot_cap, int64_t* qtile_cap,
                                    int64_t* mtile_cap) {
    if (k < 0 || C < 0) return pp::fail(PP_ERR_INVALID_ARG, "negative k (%d) or C (%d)", k, C);
    if (!slot_cap || !qtile_cap || !mtile_cap) return pp::fail(PP_ERR_INVALID_ARG, "NULL output pointer");
    *slot_cap = int64_t(k) * C;
    *qtile_cap = int64_t(k) * ceil_div(C, PP_QTILE);
    *mtile_cap = ceil_div(int64_t(k) * C, PP_MTILE);
    return PP_OK;
}

extern "C" pp_status pp_pack(const int32_t* lengths, int32_t k, int32_t capacity, pp_plan* plan) {
    pp::clear_error();
    int32_t m = 0;
    int64_t total = 0;
    if (pp_status st = check_lengths(lengths, k, &m, &total)) return st;
    if (capacity < 0) return pp::fail(PP_ERR_INVALID_ARG, "capacity %d is negative", capacity);
    const int32_t C = capacity == 0 ? m : capacity;
    if (m > C) return pp::fail(PP_ERR_TOO_LONG, "a prompt of length %d does not fit a row of %d", m, C);
    if (pp_status st = check_plan_buffers(plan, k, C)) return st;

    // First-fit decreasing over prompts sorted by (-length, index).
    std::vector<int32_t> order(k);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(),
                     [&](int32_t a, int32_t b) { return lengths[a] > lengths[b]; });
    std::vector<int32_t> room;                 // free slots per open row
    std::vector<std::vector<int32_t>> rows;    // prompts per row, placement order
    for (int32_t i : order) {
        size_t r = 0;
        while (r < room.size() && room[r] < lengths[i]) ++r;
        if (r == room.size()) {
            room.push_back(C);
            rows.emplace_back();
        }
        room[r] -= lengths[i];
        rows[r].push_back(i);
    }
    const int32_t n_rows = static_cast<int32_t>(rows.size());

    const int64_t T = int64_t(n_rows) * C;
    if (T > INT32_MAX) return pp::fail(PP_ERR_INVALID_ARG, "packed batch of %lld slots overflows int32",
                                       (long long)T);
    prefix_offsets(lengths, k, plan->prompt_kv_off);
    std::fill(plan->slot_seg, plan->slot_seg + T, -1);
    std::fill(plan->slot_pos, plan->slot_pos + T, 0);
    std::fill(plan->slot_kv, plan->slot_kv + T, -1);
    int32_t s = 0;
    plan->row_seg_ptr[0] = 0;
    for (int32_t r = 0; r < n_rows; ++r) {
        int64_t slot = int64_t(r) * C;
        for (int32_t i : rows[r]) {
            plan->seg_prompt[s] = i;
            plan->seg_start[s] = static_cast<int32_t>(slot);
            plan->seg_len[s] = lengths[i];
            const int32_t kv0 = plan->prompt_kv_off[i];
            for (int32_t j = 0; j < lengths[i]; ++j) {
                plan->slot_seg[slot + j] = s;
                plan->slot_pos[slot + j] = j;          // restart positions
                plan->slot_kv[slot + j] = kv0 + j;     // UNPACK target
            }
            slot += lengths[i];
            ++s;
        }
        plan->row_seg_ptr[r + 1] = s;
    }
    plan->k = k;
    plan->capacity = C;
    plan->n_rows = n_rows;
    plan->max_len = m;
    plan->total_len = static_cast<int32_t>(total);
    build_qtiles(plan, k);
    build_mtiles(plan, T);
    return PP_OK;
}

extern "C" pp_status pp_pack_padded(const int32_t* lengths, int32_t k, pp_plan* plan) {
    pp::clear_error();
    int32_t m = 0;
    int64_t total = 0;
    if (pp_status st = check_lengths(lengths, k, &m, &total)) return st;
    if (pp_status st = check_plan_buffers(plan, k, m)) return st;
    const int64_t T = int64_t(k) * m;
    if (T > INT32_MAX) return pp::fail(PP_ERR_INVALID_ARG, "padded batch of %lld slots overflows int32",
                                       (long long)T);
    prefix_offsets(lengths, k, plan->prompt_kv_off);
    for (int32_t i = 0; i < k; ++i) {
        const int64_t base = int64_t(i) * m;
        plan->row_seg_ptr[i] = i;
        plan->seg_prompt[i] = i;
        plan->seg_start[i] = static_cast<int32_t>(base);
        plan->seg_len[i] = m;
        for (int32_t j = 0; j < m; ++j) {
            plan->slot_seg[base + j] = i;
            plan->slot_pos[base + j] = j;
            plan->slot_kv[base + j] = j < lengths[i] ? plan->prompt_kv_off[i] + j : -1;
        }
    }
    plan->row_seg_ptr[k] = k;
    plan->k = k;
    plan->capacity = m;
    plan->n_rows = k;
    plan->max_len = m;
    plan->total_len = static_cast<int32_t>(total);
    build_qtiles(plan, k);
    build_mtiles(plan, T);
    return PP_OK;
}
