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

// Per-bundle fixed cost (epilogue, header loads) in units of one slot step.
constexpr int64_t kBundleOverhead = 3;

// Bytes of the per-bundle table (rows and biases) the strip kernel keeps in LDS.
int64_t table_bytes(const Input &in, int g) {
    const int64_t groups = 64 / g;
    const int64_t rows = in.cout / in.block_rows;
    const int64_t bundles = (rows + groups - 1) / groups;
    return ((bundles * groups * (1 + in.block_rows) * 4) + 15) & ~int64_t(15);
}

void choose_geometry(const Input &in, const Options &opt, PackedPlan &p) {
    const int e = in.storage == 1 ? 2 : 4;
    auto strip_bytes = [&](int g, int nv) { return static_cast<int64_t>(in.cin) * g * nv * kLaneBytes; };
    auto fits = [&](int g, int nv) { return strip_bytes(g, nv) + table_bytes(in, g) <= kMaxLdsBytes; };
    // Strip rows of 256 bytes: 16 lanes x one 16-byte vector read 256
    // contiguous bytes (all 64 LDS banks) per row, so the four lane groups of a
    // wavefront take four conflict-free LDS cycles.  Wider inputs fall back to
    // 128-byte rows (8 lanes), then to the direct-load kernel.
    int g = opt.lanes_per_row, nv = opt.vecs_per_lane;
    if (g == 0 && nv == 0) {
        if (fits(16, 1)) {
            g = 16;
            nv = 1;
        } else if (fits(8, 1)) {
            g = 8;
            nv = 1;
        } else {
            g = 16;
            nv = 1;
        }
    } else {
        if (g == 0)
            g = 16;
        if (nv == 0)
            nv = 1;
    }
    const bool strip = fits(g, nv);
    if (!strip)
        nv = 1;  // the direct-load kernel reads one vector per lane
    p.lanes_per_row = g;
    p.vecs_per_lane = nv;
    p.groups = 64 / g;
    p.cols_per_lane = nv * kLaneBytes / e;
    p.tile_cols = g * p.cols_per_lane;
    if (strip) {
        p.kernel = KERNEL_STRIP;
        p.strip_bytes = static_cast<int32_t>(strip_bytes(g, nv));
        p.lds_bytes = static_cast<int32_t>(strip_bytes(g, nv) + table_bytes(in, g));
        p.loader_waves = opt.prefetch
                             ? static_cast<int32_t>((strip_bytes(g, nv) + kLoaderBytesPerWave - 1) /
                                                    kLoaderBytesPerWave)
                             : 0;
    } else {
        p.kernel = KERNEL_DIRECT;
        p.strip_bytes = 0;
        p.lds_bytes = 0;
        p.loader_waves = 0;
    }
}

}  // namespace

Status build_plan(const Input &in, const Options &opt, PackedPlan &p, std::string &err) {
    Status st = validate(in, err);
    if (st != OK)
        return st;
    if (opt.lanes_per_row != 0 && opt.lanes_per_row != 8 && opt.lanes_per_row != 16 &&
        opt.lanes_per_row != 32 && opt.lanes_per_row != 64) {
        err = "lanes_per_row must be 0, 8, 16, 32 or 64";
        return E_ARG;
    }
    if (opt.waves < 0 || opt.waves > 16) {
        err = "waves must be in [0, 16]";
        return E_ARG;
    }
    if (opt.vecs_per_lane != 0 && opt.vecs_per_lane != 1 && opt.vecs_per_lane != 2) {
        err = "vecs_per_lane must be 0, 1 or 2";
        return E_ARG;
    }
    if (opt.lanes_per_row == 64 && opt.vecs_per_lane == 2) {
        err = "lanes_per_row = 64 takes one vector per lane";
        return E_ARG;
    }
    if (opt.reorder != 0 && opt.reorder != 1) {
        err = "reorder must be 0 or 1";
        return E_ARG;
    }
    if (opt.prefetch != 0 && opt.prefetch != 1) {
        err = "prefetch must be 0 or 1";
        return E_ARG;
    }

    p = PackedPlan();
    p.cout = in.cout;
    p.cin = in.cin;
    p.k = in.block_rows;
    p.act = in.act;
    p.storage = in.storage;
    choose_geometry(in, opt, p);

    const int32_t k = in.block_rows;
    const int32_t rows = in.cout / k;
    const int32_t G = p.groups;
    p.nnzb = in.row_ptr[rows];

    // 1. processing order: descending nonzero count, ties by row index (stable)
    p.perm.resize(rows);
    std::iota(p.perm.begin(), p.perm.end(), 0);
    auto len = [&](int32_t r) { return in.row_ptr[r + 1] - in.row_ptr[r]; };
    if (opt.reorder)
        std::stable_sort(p.perm.begin(), p.perm.end(), [&](int32_t a, int32_t b) { return len(a) > len(b); });

    // 2. bundles of G consecutive rows in that order
    p.row_nnz.resize(rows);
    for (int32_t r = 0; r < rows; ++r)
        p.row_nnz[r] = len(r);
    const int32_t nb = (rows + G - 1) / G;
    std::vector<int32_t> blen(nb, 0);
    for (int32_t b = 0; b < nb; ++b)
        for (int32_t g = 0; g < G && b * G + g < rows; ++g)
            blen[b] = std::max(blen[b], len(p.perm[b * G + g]));
    // padded to whole steps of 4 slots, at least one step
    for (int32_t b = 0; b < nb; ++b)
        blen[b] = std::max<int32_t>(4, (blen[b] + 3) & ~3);

    // 3. longest-processing-time-first assignment of bundles to waves
    const int32_t max_waves = kMaxWaves - p.loader_waves;
    if (opt.waves > max_waves) {
        err = "waves = " + std::to_string(opt.waves) + " plus " + std::to_string(p.loader_waves) +
              " loader waves exceeds " + std::to_string(kMaxWaves) + " wavefronts per workgroup";
        return E_ARG;
    }
    int32_t waves = opt.waves ? opt.waves : std::min<int32_t>(max_waves, std::max<int32_t>(nb, 1));
    p.waves = waves;
    std::vector<int32_t> order(nb);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return blen[a] > blen[b]; });
    using Item = std::pair<int64_t, int32_t>;  // (load, wave)
    std::priority_queue<Item, std::vector<Item>, std::greater<Item>> heap;
    for (int32_t w = 0; w < waves; ++w)
        heap.push({0, w});
    std::vector<std::vector<int32_t>> lists(waves);
    std::vector<int64_t> load(waves, 0);
    for (int32_t b : order) {
        Item it = heap.top();
        heap.pop();
        lists[it.second].push_back(b);
        it.first += blen[b] + kBundleOverhead;
        load[it.second] = it.first;
        heap.push(it);
    }
    p.max_wave_cost = waves ? *std::max_element(load.begin(), load.end()) : 0;
    p.sum_wave_cost = std::accumulate(load.begin(), load.end(), int64_t(0));

    // 4. pack, bundles stored in wave order; every bundle is a whole number
    // of steps (4 slots per lane group) and at least one step long
    p.wave_ptr.assign(waves + 1, 0);
    p.hdr.reserve(4 * static_cast<size_t>(nb));
    p.rows.reserve(static_cast<size_t>(G) * nb);
    p.bundle_bias.reserve(static_cast<size_t>(G) * nb * k);
    int64_t slot = 0;
    for (int32_t w = 0; w < waves; ++w) {
        for (int32_t b : lists[w]) {
            const int32_t L = blen[b];
            if (slot + static_cast<int64_t>(L) * G > (int64_t(1) << 30)) {
                err = "packed plan too large";
                return E_SHAPE;
            }
            p.hdr.push_back(static_cast<int32_t>(slot));
            p.hdr.push_back(L / 4);
            p.hdr.push_back(0);
            p.hdr.push_back(0);
            const size_t need = static_cast<size_t>(slot + static_cast<int64_t>(L) * G);
            p.idx.resize(need, 0);
            p.val.resize(need * k, 0.0f);
            for (int32_t g = 0; g < G; ++g) {
                const int32_t pos = b * G + g;
                const int32_t rb = pos < rows ? p.perm[pos] : -1;
                p.rows.push_back(rb);
                for (int32_t i = 0; i < k; ++i)
                    p.bundle_bias.push_back(rb >= 0 && in.bias ? in.bias[rb * k + i] : 0.0f);
                // the last step of the bundle is marked in its first slot
                p.idx[slot + (static_cast<int64_t>(L / 4 - 1) * G + g) * 4] |= kLastStepFlag;
                if (rb < 0)
                    continue;
                const int32_t s0 = in.row_ptr[rb];
                const int32_t n = len(rb);
                for (int32_t t = 0; t < n; ++t) {
                    const int64_t sl = slot + (static_cast<int64_t>(t >> 2) * G + g) * 4 + (t & 3);
                    p.idx[sl] = (p.idx[sl] & kLastStepFlag) | in.col_idx[s0 + t];
                    for (int32_t i = 0; i < k; ++i) {
                        float v = in.values[static_cast<int64_t>(s0 + t) * k + i];
                        if (in.storage == 1)
                            v = half_to_float(float_to_half_rne(v));
                        p.val[sl * k + i] = v;
                    }
                }
            }
            slot += static_cast<int64_t>(L) * G;
        }
        p.wave_ptr[w + 1] = static_cast<int32_t>(p.hdr.size() / 4);
    }
    // Keep every stream a whole number of 16-byte vectors and leave
    // kLookaheadSteps main-loop steps (4 slots per lane group each) of padding
    // after the last bundle: the kernel fetches slots of later steps before it
    // knows whether the bundle continues.
    slot = ((slot + 3) & ~int64_t(3)) + (kLookaheadSteps + 1) * 4 * static_cast<int64_t>(G) + 4;
    p.idx.resize(static_cast<size_t>(slot), 0);
    p.val.resize(static_cast<size_t>(slot) * k, 0.0f);
    p.slots = slot;
    if (p.hdr.empty())
        p.hdr.assign(4, 0);
    // LDS copy of the per-bundle rows and biases, after the strip
    p.meta_bytes = static_cast<int32_t>(p.rows.size() * sizeof(int32_t) + p.bundle_bias.size() * sizeof(float));

    p.bias.assign(in.cout, 0.0f);
    if (in.bias)
        std::copy(in.bias, in.bias + in.cout, p.bias.begin());
    return OK;
}

void unpack_plan(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, int32_t *perm) {
    const int32_t k = p.k;
    const int32_t rows = p.cout / k;
    const int32_t G = p.groups;
    std::vector<std::vector<int32_t>> cols(rows);
    std::vector<std::vector<float>> vals(rows);
    const int32_t nb = static_cast<int32_t>(p.wave_ptr.back());
    // each row's real entries are the first row_nnz[rb] slots of its sequence
    for (int32_t b = 0; b < nb; ++b) {
        const int64_t S = p.hdr[4 * b];
        for (int32_t g = 0; g < G; ++g) {
            const int32_t rb = p.rows[static_cast<size_t>(b) * G + g];
            if (rb < 0)
                continue;
            for (int32_t t = 0; t < p.row_nnz[rb]; ++t) {
                const int64_t sl = S + (static_cast<int64_t>(t >> 2) * G + g) * 4 + (t & 3);
                cols[rb].push_back(p.idx[sl] & ~kLastStepFlag);
                for (int32_t i = 0; i < k; ++i)
                    vals[rb].push_back(p.val[sl * k + i]);
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
