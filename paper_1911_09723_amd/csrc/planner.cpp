// Host-side format planner: validation, row ordering, bundling, wave
// balancing and packing.  See planner.hpp for the packed layout.
#include "planner.hpp"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <numeric>
#include <queue>
#include <sstream>

namespace spconv {

uint16_t float_to_half_rne(float v) {
    uint32_t f;
    std::memcpy(&f, &v, 4);
    const uint32_t sign = (f >> 16) & 0x8000u;
    const uint32_t a = f & 0x7fffffffu;
    if (a >= 0x7f800000u)  // infinity or NaN
        return static_cast<uint16_t>(sign | (a > 0x7f800000u ? 0x7e00u : 0x7c00u));
    if (a >= 0x477ff000u)  // >= 65520: rounds past the largest finite half (65504)
        return static_cast<uint16_t>(sign | 0x7c00u);
    if (a >= 0x38800000u) {  // normal half range, |v| >= 2^-14
        const uint32_t m = a - 0x38000000u;  // exponent bias 127 -> 15
        uint32_t r = m >> 13;
        const uint32_t rem = m & 0x1fffu;
        if (rem > 0x1000u || (rem == 0x1000u && (r & 1u)))
            ++r;  // a mantissa carry correctly bumps the exponent
        return static_cast<uint16_t>(sign | r);
    }
    if (a < 0x33000000u)  // below 2^-25: rounds to zero (2^-25 itself ties to even zero)
        return static_cast<uint16_t>(sign);
    // subnormal half: value = mant * 2^(e - 150); in units of 2^-24 that is mant >> (126 - e)
    const uint32_t e = a >> 23;
    const uint32_t mant = (a & 0x7fffffu) | 0x800000u;
    const uint32_t shift = 126u - e;
    uint32_t r = mant >> shift;
    const uint32_t rem = mant & ((1u << shift) - 1u);
    const uint32_t half = 1u << (shift - 1u);
    if (rem > half || (rem == half && (r & 1u)))
        ++r;
    return static_cast<uint16_t>(sign | r);
}

float half_to_float(uint16_t h) {
    const int sign = (h >> 15) & 1;
    const int expo = (h >> 10) & 0x1f;
    const int frac = h & 0x3ff;
    float v;
    if (expo == 0)
        v = std::ldexp(static_cast<float>(frac), -24);
    else if (expo == 31)
        v = frac ? NAN : INFINITY;
    else
        v = std::ldexp(static_cast<float>(frac | 0x400), expo - 25);
    return sign ? -v : v;
}

Status validate(const Input &in, std::string &err) {
    std::ostringstream os;
    if (in.act < 0 || in.act > 2) {
        err = "act must be SPCONV_ACT_NONE, _RELU or _RELU6";
        return E_ARG;
    }
    if (in.storage < 0 || in.storage > 1) {
        err = "storage must be SPCONV_F32 or SPCONV_F16";
        return E_ARG;
    }
    if (in.block_rows <= 0) {
        err = "block_rows must be positive";
        return E_ARG;
    }
    if (in.block_rows != 1 && in.block_rows != 4) {
        os << "block_rows = " << in.block_rows << " is not supported (1 or 4)";
        err = os.str();
        return E_UNSUPPORTED;
    }
    if (in.cout <= 0 || in.cin <= 0) {
        os << "cout and cin must be >= 1 (got cout = " << in.cout << ", cin = " << in.cin << ")";
        err = os.str();
        return E_SHAPE;
    }
    if (in.cout % in.block_rows) {
        os << "cout = " << in.cout << " is not a multiple of block_rows = " << in.block_rows;
        err = os.str();
        return E_SHAPE;
    }
    if (in.cin > (1 << 24)) {
        err = "cin must be at most 2^24";
        return E_SHAPE;
    }
    if (!in.row_ptr) {
        err = "row_ptr is NULL";
        return E_ARG;
    }
    const int32_t rows = in.cout / in.block_rows;
    if (in.row_ptr[0] != 0) {
        os << "row_ptr[0] = " << in.row_ptr[0] << ", expected 0";
        err = os.str();
        return E_FORMAT;
    }
    for (int32_t r = 0; r < rows; ++r) {
        if (in.row_ptr[r + 1] < in.row_ptr[r]) {
            os << "row_ptr decreases at block row " << r << " (" << in.row_ptr[r] << " -> "
               << in.row_ptr[r + 1] << ")";
            err = os.str();
            return E_FORMAT;
        }
        if (in.row_ptr[r + 1] - in.row_ptr[r] > in.cin) {
            os << "block row " << r << " has " << (in.row_ptr[r + 1] - in.row_ptr[r])
               << " entries but cin = " << in.cin;
            err = os.str();
            return E_FORMAT;
        }
    }
    const int64_t nnzb = in.row_ptr[rows];
    if (nnzb > 0 && (!in.col_idx || !in.values)) {
        err = "col_idx or values is NULL but the matrix has stored entries";
        return E_ARG;
    }
    if (nnzb * static_cast<int64_t>(in.block_rows) > (int64_t(1) << 30)) {
        err = "too many stored values (limit 2^30)";
        return E_SHAPE;
    }
    for (int32_t r = 0; r < rows; ++r) {
        for (int32_t t = in.row_ptr[r]; t < in.row_ptr[r + 1]; ++t) {
            const int32_t c = in.col_idx[t];
            if (c < 0 || c >= in.cin) {
                os << "col_idx[" << t << "] = " << c << " is outside [0, " << in.cin << ") in block row " << r;
                err = os.str();
                return E_FORMAT;
            }
            if (t > in.row_ptr[r] && c <= in.col_idx[t - 1]) {
                os << "col_idx not strictly ascending in block row " << r << " at entry " << t << " ("
                   << in.col_idx[t - 1] << ", " << c << ")";
                err = os.str();
                return E_FORMAT;
            }
        }
    }
    for (int64_t i = 0; i < nnzb * in.block_rows; ++i) {
        if (!std::isfinite(in.values[i])) {
            os << "values[" << i << "] is not finite";
            err = os.str();
            return E_FORMAT;
        }
    }
    if (in.bias) {
        for (int32_t r = 0; r < in.cout; ++r) {
            if (!std::isfinite(in.bias[r])) {
                os << "bias[" << r << "] is not finite";
                err = os.str();
                return E_FORMAT;
            }
        }
    }
    return OK;
}

namespace {

// Per-bundle fixed cost (epilogue, table reads) in units of one slot.
constexpr int64_t kBundleOverhead = 3;
// Most fp32 accumulators one lane may hold (k rows x its columns), and the
// most the automatic choice uses (a 1xk block's k weights per slot also sit
// in the lane's registers, so wider blocks take narrower column sets).
constexpr int32_t kMaxAccumulators = 64;
constexpr int32_t kAutoAccumulators = 32;

int32_t bundles_of(int32_t rows, int32_t nb) { return (rows + nb - 1) / nb; }

// Bytes of the per-bundle table the kernels keep in LDS, 16-byte rounded.
int64_t table_bytes(int32_t nbundles, int32_t nb, int32_t k) {
    return (static_cast<int64_t>(nbundles) * nb * (1 + k) * 4 + 15) & ~int64_t(15);
}

Status choose_geometry(const Input &in, const Options &opt, PackedPlan &p, std::string &err) {
    const int32_t e = in.storage == 1 ? 2 : 4;
    const int32_t k = in.block_rows;
    const int32_t rows = in.cout / k;
    auto accumulators = [&](int32_t g) { return k * (16 / g) * (16 / e); };
    int32_t g = opt.group_lanes;
    if (g == 0) {
        // 4 lanes per row (16 bytes of X per lane and slot, 4 vectors) unless
        // the accumulators would not fit; wider groups when there are too few
        // bundles to occupy the workgroup's wavefronts
        g = 4;
        while (g < 16 && accumulators(g) > kAutoAccumulators)
            g *= 2;
        while (g < 16 && bundles_of(rows, 64 / g) < 8)
            g *= 2;
    } else if (accumulators(g) > kMaxAccumulators) {
        err = "group_lanes = " + std::to_string(g) + " needs " + std::to_string(accumulators(g)) +
              " accumulators per lane (limit " + std::to_string(kMaxAccumulators) + ")";
        return E_UNSUPPORTED;
    }
    p.group_lanes = g;
    p.bundle_rows = 64 / g;
    p.cols_per_lane = (16 / g) * (16 / e);
    p.tile_cols = kRowBytes / e;
    const int32_t nbundles = bundles_of(rows, p.bundle_rows);
    const int64_t table = table_bytes(nbundles, p.bundle_rows, k) + kCtlBytes;
    const int32_t strip_rows = (in.cin + 3) / 4 * 4;
    const int64_t strip = static_cast<int64_t>(strip_rows) * kRowBytes;
    const bool fits = strip + table <= kMaxLdsBytes;
    if (opt.kernel == 1 && !fits) {
        err = "the X strip of cin = " + std::to_string(in.cin) + " channels does not fit in LDS";
        return E_UNSUPPORTED;
    }
    if (table > kMaxLdsBytes) {
        err = "the bundle table of cout = " + std::to_string(in.cout) + " rows does not fit in LDS";
        return E_UNSUPPORTED;
    }
    if (opt.kernel != 2 && fits) {
        p.kernel = KERNEL_STRIP;
        p.row_scale = kRowBytes;
        p.strip_rows = strip_rows;
        p.split_rows = (strip_rows / 4 + 1) / 2 * 4;
        p.lds_bytes = static_cast<int32_t>(strip + table);
    } else {
        p.kernel = KERNEL_DIRECT;
        p.row_scale = 1;
        p.strip_rows = 0;
        p.lds_bytes = static_cast<int32_t>(table);
    }
    return OK;
}

}  // namespace

Status build_plan(const Input &in, const Options &opt, PackedPlan &p, std::string &err) {
    Status st = validate(in, err);
    if (st != OK)
        return st;
    if (opt.kernel < 0 || opt.kernel > 2) {
        err = "kernel must be 0 (automatic), 1 (strip) or 2 (direct)";
        return E_ARG;
    }
    if (opt.group_lanes != 0 && opt.group_lanes != 4 && opt.group_lanes != 8 && opt.group_lanes != 16) {
        err = "group_lanes must be 0, 4, 8 or 16";
        return E_ARG;
    }
    if (opt.waves < 0 || opt.waves > kMaxWaves) {
        err = "waves must be in [0, 16]";
        return E_ARG;
    }
    if (opt.reorder != 0 && opt.reorder != 1) {
        err = "reorder must be 0 or 1";
        return E_ARG;
    }

    p = PackedPlan();
    p.cout = in.cout;
    p.cin = in.cin;
    p.k = in.block_rows;
    p.act = in.act;
    p.storage = in.storage;
    st = choose_geometry(in, opt, p, err);
    if (st != OK)
        return st;

    const int32_t k = in.block_rows;
    const int32_t rows = in.cout / k;
    const int32_t NB = p.bundle_rows;
    p.nnzb = in.row_ptr[rows];

    // 1. processing order: descending nonzero count, ties by row index (stable)
    p.perm.resize(rows);
    std::iota(p.perm.begin(), p.perm.end(), 0);
    auto len = [&](int32_t r) { return in.row_ptr[r + 1] - in.row_ptr[r]; };
    if (opt.reorder)
        std::stable_sort(p.perm.begin(), p.perm.end(), [&](int32_t a, int32_t b) { return len(a) > len(b); });

    // 2. bundles of NB consecutive rows in that order, each a whole number of
    // steps of 4 slots and at least one step long
    p.row_nnz.resize(rows);
    for (int32_t r = 0; r < rows; ++r)
        p.row_nnz[r] = len(r);
    const int32_t nb = bundles_of(rows, NB);
    std::vector<int32_t> bsteps(nb, 0);
    for (int32_t b = 0; b < nb; ++b) {
        int32_t l = 0;
        for (int32_t q = 0; q < NB && b * NB + q < rows; ++q)
            l = std::max(l, len(p.perm[b * NB + q]));
        bsteps[b] = std::max<int32_t>(1, (l + kStepSlots - 1) / kStepSlots);
    }

    // 3. longest-processing-time-first assignment of bundles to waves
    const int32_t waves = opt.waves ? opt.waves : std::min<int32_t>(kMaxWaves, nb);
    p.waves = waves;
    std::vector<int32_t> order(nb);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return bsteps[a] > bsteps[b]; });
    using Item = std::pair<int64_t, int32_t>;  // (load, wave)
    std::priority_queue<Item, std::vector<Item>, std::greater<Item>> heap;
    for (int32_t w = 0; w < waves; ++w)
        heap.push({0, w});
    std::vector<std::vector<int32_t>> lists(waves);
    std::vector<int64_t> load(waves, 0);
    std::vector<int32_t> rank_of(nb, 0);
    for (int32_t i = 0; i < nb; ++i) {
        const int32_t b = order[i];
        rank_of[b] = i;
        Item it = heap.top();
        heap.pop();
        lists[it.second].push_back(b);
        it.first += kStepSlots * static_cast<int64_t>(bsteps[b]) + kBundleOverhead;
        load[it.second] = it.first;
        heap.push(it);
    }
    p.max_wave_cost = waves ? *std::max_element(load.begin(), load.end()) : 0;
    p.sum_wave_cost = std::accumulate(load.begin(), load.end(), int64_t(0));

    // 4. pack: bundles in wave order, each wave's bundles one continuous stream
    int64_t total_steps = 0;
    for (int32_t b = 0; b < nb; ++b)
        total_steps += bsteps[b];
    if (total_steps * NB * kStepSlots * k * 4 >= (int64_t(1) << 31)) {
        err = "packed plan too large";
        return E_SHAPE;
    }
    const int32_t pad_channel = p.kernel == KERNEL_STRIP ? p.strip_rows - 1 : 0;
    p.idx.assign(static_cast<size_t>(total_steps * NB * kStepSlots), pad_channel * p.row_scale);
    p.val.assign(static_cast<size_t>(total_steps * NB * kStepSlots * k), 0.0f);
    p.wave_ptr.assign(waves + 1, 0);
    p.hdr.reserve(2 * static_cast<size_t>(nb));
    p.rows.reserve(static_cast<size_t>(NB) * nb);
    p.bundle_bias.reserve(static_cast<size_t>(NB) * nb * k);
    p.rank.reserve(nb);
    p.wave_meta.assign(2 * static_cast<size_t>(waves), 0);
    // slots of a row that read the strip's lower part (ascending channels)
    auto lower = [&](int32_t rb) {
        int32_t n = 0;
        while (n < len(rb) && in.col_idx[in.row_ptr[rb] + n] < p.split_rows)
            ++n;
        return n;
    };
    int64_t step = 0;   // first step of the next bundle
    int32_t bglob = 0;  // bundles packed so far
    for (int32_t w = 0; w < waves; ++w) {
        const int64_t wstart = step;
        int64_t rel0 = 0, need1 = -1;
        for (int32_t b : lists[w]) {
            // a0: steps until every row has passed its lower-part channels;
            // a1: first step in which some row reads the upper part (a padding
            // group or a row's padding slots do from their first slot)
            int64_t a0 = 0, a1 = bsteps[b];
            for (int32_t q = 0; q < NB; ++q) {
                const int32_t pos = b * NB + q;
                const int32_t n0 = pos < rows ? lower(p.perm[pos]) : 0;
                const int32_t n = pos < rows ? len(p.perm[pos]) : 0;
                a0 = std::max<int64_t>(a0, (n0 + kStepSlots - 1) / kStepSlots);
                if (n0 < static_cast<int64_t>(bsteps[b]) * kStepSlots && (n0 < n || n < bsteps[b] * kStepSlots))
                    a1 = std::min<int64_t>(a1, n0 / kStepSlots);
            }
            rel0 = std::max(rel0, step - wstart + a0);
            if (a1 < bsteps[b] && need1 < 0)
                need1 = step - wstart + a1;
            p.hdr.push_back(static_cast<int32_t>(step));
            p.hdr.push_back(bsteps[b]);
            p.rank.push_back(rank_of[b]);
            for (int32_t q = 0; q < NB; ++q) {
                const int32_t pos = b * NB + q;
                const int32_t rb = pos < rows ? p.perm[pos] : -1;
                p.rows.push_back(rb);
                for (int32_t i = 0; i < k; ++i)
                    p.bundle_bias.push_back(rb >= 0 && in.bias ? in.bias[rb * k + i] : 0.0f);
                if (rb < 0)
                    continue;
                const int32_t r0 = in.row_ptr[rb];
                for (int32_t t = 0; t < len(rb); ++t) {
                    const int64_t e = ((step + t / kStepSlots) * NB + q) * kStepSlots + t % kStepSlots;
                    p.idx[e] = in.col_idx[r0 + t] * p.row_scale;
                    for (int32_t i = 0; i < k; ++i) {
                        float v = in.values[static_cast<int64_t>(r0 + t) * k + i];
                        if (in.storage == 1)
                            v = half_to_float(float_to_half_rne(v));
                        p.val[e * k + i] = v;
                    }
                }
            }
            step += bsteps[b];
            ++bglob;
        }
        p.wave_ptr[w + 1] = bglob;
        p.wave_meta[2 * w] = static_cast<int32_t>(rel0);
        p.wave_meta[2 * w + 1] = static_cast<int32_t>(need1 < 0 ? step - wstart : need1);
        if (!lists[w].empty())
            ++p.busy_waves;
    }
    p.slots = total_steps * NB * kStepSlots;
    p.max_parts = 1;
    while (p.max_parts * 2 <= std::min<int32_t>(kMaxParts, nb))
        p.max_parts *= 2;
    return OK;
}

void unpack_plan(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, int32_t *perm) {
    const int32_t k = p.k;
    const int32_t rows = p.cout / k;
    const int32_t NB = p.bundle_rows;
    std::vector<std::vector<int32_t>> cols(rows);
    std::vector<std::vector<float>> vals(rows);
    // each row's real entries are the first row_nnz[rb] slots of its sequence
    for (int32_t b = 0; b < p.nbundles(); ++b) {
        const int64_t s_first = p.hdr[2 * b];
        for (int32_t q = 0; q < NB; ++q) {
            const int32_t rb = p.rows[static_cast<size_t>(b) * NB + q];
            if (rb < 0)
                continue;
            for (int32_t t = 0; t < p.row_nnz[rb]; ++t) {
                const int64_t e = ((s_first + t / kStepSlots) * NB + q) * kStepSlots + t % kStepSlots;
                cols[rb].push_back(p.idx[e] / p.row_scale);
                for (int32_t i = 0; i < k; ++i)
                    vals[rb].push_back(p.val[e * k + i]);
            }
        }
    }
    int32_t acc = 0;
    if (row_ptr)
        row_ptr[0] = 0;
    for (int32_t r = 0; r < rows; ++r) {
        if (col_idx)
            std::copy(cols[r].begin(), cols[r].end(), col_idx + acc);
        if (values)
            std::copy(vals[r].begin(), vals[r].end(), values + static_cast<int64_t>(acc) * k);
        acc += static_cast<int32_t>(cols[r].size());
        if (row_ptr)
            row_ptr[r + 1] = acc;
    }
    if (perm)
        std::copy(p.perm.begin(), p.perm.end(), perm);
}

}  // namespace spconv
