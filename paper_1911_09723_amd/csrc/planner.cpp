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
    if (in.block_rows != 1 && in.block_rows != 2 && in.block_rows != 4) {
        os << "block_rows = " << in.block_rows << " is not supported (1, 2 or 4)";
        err = os.str();
        return E_UNSUPPORTED;
    }
    if (in.block_cols <= 0) {
        err = "block_cols must be positive";
        return E_ARG;
    }
    if (in.block_cols != 1 && in.block_cols != 2 && in.block_cols != 4) {
        os << "block_cols = " << in.block_cols << " is not supported (1, 2 or 4)";
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
    const int32_t kc = in.block_cols;
    if (nnzb * static_cast<int64_t>(in.block_rows) * kc > (int64_t(1) << 30)) {
        err = "too many stored values (limit 2^30)";
        return E_SHAPE;
    }
    for (int32_t r = 0; r < rows; ++r) {
        for (int32_t t = in.row_ptr[r]; t < in.row_ptr[r + 1]; ++t) {
            const int32_t c = in.col_idx[t];
            if (c < 0 || static_cast<int64_t>(c) + kc > in.cin) {
                os << "col_idx[" << t << "] = " << c;
                if (kc > 1)
                    os << " (a block of " << kc << " input channels)";
                os << " is outside [0, " << in.cin << ") in block row " << r;
                err = os.str();
                return E_FORMAT;
            }
            if (t > in.row_ptr[r] && c < in.col_idx[t - 1] + kc) {
                os << "col_idx not strictly ascending" << (kc > 1 ? " (blocks overlap)" : "") << " in block row "
                   << r << " at entry " << t << " (" << in.col_idx[t - 1] << ", " << c << ")";
                err = os.str();
                return E_FORMAT;
            }
        }
    }
    for (int64_t i = 0; i < nnzb * in.block_rows * kc; ++i) {
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

Status check_dense(int32_t cout, int32_t cin, const float *dense, std::string &err) {
    if (cout <= 0 || cin <= 0) {
        err = "cout and cin must be >= 1 (got cout = " + std::to_string(cout) + ", cin = " + std::to_string(cin) + ")";
        return E_SHAPE;
    }
    if (cin > (1 << 24)) {
        err = "cin must be at most 2^24";
        return E_SHAPE;
    }
    if (!dense) {
        err = "dense is NULL";
        return E_ARG;
    }
    const int64_t n = static_cast<int64_t>(cout) * cin;
    for (int64_t i = 0; i < n; ++i) {
        if (!std::isfinite(dense[i])) {
            err = "dense[" + std::to_string(i / cin) + "][" + std::to_string(i % cin) + "] is not finite";
            return E_FORMAT;
        }
    }
    return OK;
}

}  // namespace

Status detect_block_rows(int32_t cout, int32_t cin, const float *dense, int32_t &k, std::string &err) {
    const Status st = check_dense(cout, cin, dense, err);
    if (st != OK)
        return st;
    for (int32_t cand : {4, 2}) {
        if (cout % cand)
            continue;
        bool blocked = true;
        for (int32_t rb = 0; blocked && rb < cout / cand; ++rb) {
            const float *w0 = dense + static_cast<int64_t>(rb) * cand * cin;
            for (int32_t i = 1; blocked && i < cand; ++i) {
                const float *wi = w0 + static_cast<int64_t>(i) * cin;
                for (int32_t c = 0; c < cin; ++c) {
                    if ((w0[c] != 0.0f) != (wi[c] != 0.0f)) {
                        blocked = false;
                        break;
                    }
                }
            }
        }
        if (blocked) {
            k = cand;
            return OK;
        }
    }
    k = 1;
    return OK;
}

Status detect_blocks(int32_t cout, int32_t cin, const float *dense, int32_t &kr, int32_t &kc, std::string &err) {
    const Status st = check_dense(cout, cin, dense, err);
    if (st != OK)
        return st;
    // most weights per block first; on a tie, output-channel blocks (their
    // kernels reuse each X vector for every row of the block)
    static const int32_t cands[][2] = {{4, 4}, {4, 2}, {2, 4}, {4, 1}, {2, 2}, {1, 4}, {2, 1}, {1, 2}};
    for (const auto &cd : cands) {
        const int32_t r = cd[0], q = cd[1];
        if (cout % r || cin % q)
            continue;
        bool uniform = true;
        for (int32_t rb = 0; uniform && rb < cout / r; ++rb)
            for (int32_t cb = 0; uniform && cb < cin / q; ++cb) {
                const bool first = dense[static_cast<int64_t>(rb) * r * cin + static_cast<int64_t>(cb) * q] != 0.0f;
                for (int32_t i = 0; uniform && i < r; ++i)
                    for (int32_t j = 0; j < q; ++j)
                        if ((dense[(static_cast<int64_t>(rb) * r + i) * cin + cb * q + j] != 0.0f) != first) {
                            uniform = false;
                            break;
                        }
            }
        if (uniform) {
            kr = r;
            kc = q;
            return OK;
        }
    }
    kr = kc = 1;
    return OK;
}

Status dense_to_blocks(int32_t cout, int32_t cin, const float *dense, int32_t k, int32_t kc, int32_t *row_ptr,
                       int32_t *col_idx, float *values, int64_t capacity, int64_t &nnzb, std::string &err) {
    nnzb = 0;
    Status st = check_dense(cout, cin, dense, err);
    if (st != OK)
        return st;
    if (k != 1 && k != 2 && k != 4) {
        err = "block_rows = " + std::to_string(k) + " is not supported (1, 2 or 4)";
        return k <= 0 ? E_ARG : E_UNSUPPORTED;
    }
    if (kc != 1 && kc != 2 && kc != 4) {
        err = "block_cols = " + std::to_string(kc) + " is not supported (1, 2 or 4)";
        return kc <= 0 ? E_ARG : E_UNSUPPORTED;
    }
    if (cout % k) {
        err = "cout = " + std::to_string(cout) + " is not a multiple of block_rows = " + std::to_string(k);
        return E_SHAPE;
    }
    if (cin % kc) {
        err = "cin = " + std::to_string(cin) + " is not a multiple of block_cols = " + std::to_string(kc);
        return E_SHAPE;
    }
    const bool write = col_idx != nullptr;
    if (write && (!row_ptr || !values)) {
        err = "row_ptr and values must be given with col_idx";
        return E_ARG;
    }
    auto at = [&](int32_t rb, int32_t i, int32_t cb, int32_t j) {
        return dense[(static_cast<int64_t>(rb) * k + i) * cin + static_cast<int64_t>(cb) * kc + j];
    };
    auto stored = [&](int32_t rb, int32_t cb) {
        for (int32_t i = 0; i < k; ++i)
            for (int32_t j = 0; j < kc; ++j)
                if (at(rb, i, cb, j) != 0.0f)
                    return true;
        return false;
    };
    int64_t total = 0;
    for (int32_t rb = 0; rb < cout / k; ++rb)
        for (int32_t cb = 0; cb < cin / kc; ++cb)
            total += stored(rb, cb) ? 1 : 0;
    nnzb = total;
    if (total * k * kc > (int64_t(1) << 30)) {
        err = "too many stored values (limit 2^30)";
        return E_SHAPE;
    }
    if (!write) {
        if (row_ptr) {
            // row offsets only
            int32_t acc = 0;
            row_ptr[0] = 0;
            for (int32_t rb = 0; rb < cout / k; ++rb) {
                for (int32_t cb = 0; cb < cin / kc; ++cb)
                    acc += stored(rb, cb) ? 1 : 0;
                row_ptr[rb + 1] = acc;
            }
        }
        return OK;
    }
    if (total > capacity) {
        err = "capacity of " + std::to_string(capacity) + " blocks is below the " + std::to_string(total) +
              " blocks of the weight";
        return E_ARG;
    }
    int32_t t = 0;
    row_ptr[0] = 0;
    for (int32_t rb = 0; rb < cout / k; ++rb) {
        for (int32_t cb = 0; cb < cin / kc; ++cb) {
            if (!stored(rb, cb))
                continue;
            col_idx[t] = cb * kc;
            for (int32_t i = 0; i < k; ++i)
                for (int32_t j = 0; j < kc; ++j)
                    values[(static_cast<int64_t>(t) * k + i) * kc + j] = at(rb, i, cb, j);
            ++t;
        }
        row_ptr[rb + 1] = t;
    }
    return OK;
}

Status dense_to_bcsr(int32_t cout, int32_t cin, const float *dense, int32_t k, int32_t *row_ptr,
                     int32_t *col_idx, float *values, int64_t capacity, int64_t &nnzb, std::string &err) {
    return dense_to_blocks(cout, cin, dense, k, 1, row_ptr, col_idx, values, capacity, nnzb, err);
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
    // the strip and the row of zeros that padding slots read
    const int64_t strip = static_cast<int64_t>(strip_rows + 1) * kRowBytes;
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
        p.lds_bytes = static_cast<int32_t>(strip + table);
    } else {
        p.kernel = KERNEL_DIRECT;
        p.row_scale = 1;
        p.strip_rows = 0;
        p.lds_bytes = static_cast<int32_t>(table);
        if (opt.group_lanes == 0 && g != 16) {
            // the direct kernel waits on X loads from L2: 16 lanes per row (one
            // vector per lane) need the fewest registers, so more wavefronts
            // stay resident, and give 4x more bundles to spread
            g = 16;
            p.group_lanes = g;
            p.bundle_rows = 64 / g;
            p.cols_per_lane = (16 / g) * (16 / e);
            const int64_t t16 = table_bytes(bundles_of(rows, p.bundle_rows), p.bundle_rows, k) + kCtlBytes;
            if (t16 > kMaxLdsBytes) {
                err = "the bundle table of cout = " + std::to_string(in.cout) + " rows does not fit in LDS";
                return E_UNSUPPORTED;
            }
            p.lds_bytes = static_cast<int32_t>(t16);
        }
    }
    return OK;
}

// The strip parts each channel of a step reads, as a bit mask, and the
// step's merge key (lowest + highest channel it reads; padding reads none).
struct StepReads {
    uint32_t regions = 0;
    int64_t key = 0;
};

StepReads step_reads(const PackedPlan &p, int64_t step) {
    const int64_t rec = static_cast<int64_t>(p.bundle_rows) * kStepSlots;
    StepReads r;
    int32_t lo = INT32_MAX, hi = -1;
    for (int64_t e = step * rec; e < (step + 1) * rec; ++e) {
        const int32_t c = p.idx[e] / p.row_scale;
        if (c >= p.strip_rows)
            continue;  // padding: the row of zeros
        lo = std::min(lo, c);
        hi = std::max(hi, c);
        r.regions |= 1u << (c / p.region_rows);
    }
    r.key = hi < 0 ? 0 : static_cast<int64_t>(lo) + hi;
    return r;
}

// Interleaved streams, selector words and region events (planner.hpp).
void build_interleaved(PackedPlan &p) {
    const int32_t NB = p.bundle_rows, k = p.k, S = p.pipe_sets;
    const int64_t rec = static_cast<int64_t>(NB) * kStepSlots;
    p.pidx.assign(p.idx.size(), 0);
    p.pval.assign(p.val.size(), 0.0f);
    p.psel.clear();
    p.sel_ptr.assign(p.waves + 1, 0);
    p.wave_ev.assign(static_cast<size_t>(p.waves) * kWaveEvents, INT32_MAX);
    for (int32_t w = 0; w < p.waves; ++w) {
        const int32_t b0 = p.wave_ptr[w], b1 = p.wave_ptr[w + 1];
        p.sel_ptr[w + 1] = p.sel_ptr[w];
        if (b0 == b1)
            continue;
        const int64_t ws0 = p.hdr[2 * b0];
        // merge each set group's steps by key, each bundle's steps in order
        std::vector<int64_t> src;
        std::vector<uint32_t> bits;
        for (int32_t g = b0; g < b1; g += S) {
            const int32_t ng = std::min(S, b1 - g);
            std::vector<int32_t> next(ng, 0);
            for (;;) {
                int32_t best = -1;
                int64_t best_key = 0;
                for (int32_t i = 0; i < ng; ++i) {
                    const int32_t b = g + i;
                    if (next[i] == p.hdr[2 * b + 1])
                        continue;
                    const int64_t key = step_reads(p, p.hdr[2 * b] + next[i]).key;
                    if (best < 0 || key < best_key) {
                        best = i;
                        best_key = key;
                    }
                }
                if (best < 0)
                    break;
                const int32_t b = g + best;
                src.push_back(p.hdr[2 * b] + next[best]);
                ++next[best];
                bits.push_back(static_cast<uint32_t>(best) | (next[best] == p.hdr[2 * b + 1] ? 2u : 0u));
            }
        }
        const int64_t len = static_cast<int64_t>(src.size());
        std::vector<int64_t> need(kMaxRegions, INT64_MAX), rel(kMaxRegions, -1);
        for (int64_t i = 0; i < len; ++i) {
            const int64_t d = ws0 + i;
            std::copy(p.idx.begin() + src[i] * rec, p.idx.begin() + (src[i] + 1) * rec, p.pidx.begin() + d * rec);
            std::copy(p.val.begin() + src[i] * rec * k, p.val.begin() + (src[i] + 1) * rec * k,
                      p.pval.begin() + d * rec * k);
            const uint32_t m = step_reads(p, src[i]).regions;
            for (int32_t q = 0; q < p.regions; ++q)
                if (m >> q & 1u) {
                    need[q] = std::min(need[q], i);
                    rel[q] = i;
                }
        }
        const int64_t words = (len + kSelSteps - 1) / kSelSteps;
        const size_t base = p.psel.size();
        p.psel.resize(base + words, 0u);
        for (int64_t i = 0; i < len; ++i)
            p.psel[base + i / kSelSteps] |= bits[i] << (2 * (i % kSelSteps));
        p.sel_ptr[w + 1] = static_cast<int32_t>(p.psel.size());
        std::vector<int32_t> ne, re;
        for (int32_t q = 0; q < p.regions; ++q) {
            if (need[q] != INT64_MAX)
                ne.push_back(static_cast<int32_t>(need[q] << 4 | q));
            re.push_back(static_cast<int32_t>((rel[q] < 0 ? 0 : rel[q]) << 4 | q));
        }
        std::sort(ne.begin(), ne.end());
        std::sort(re.begin(), re.end());
        std::copy(ne.begin(), ne.end(), p.wave_ev.begin() + static_cast<size_t>(w) * kWaveEvents);
        std::copy(re.begin(), re.end(), p.wave_ev.begin() + static_cast<size_t>(w) * kWaveEvents + kMaxRegions);
    }
}

}  // namespace

// The fused depthwise stage's arguments: fp32 storage, the strip kernel,
// stride 1 or 2, finite taps and biases.
static Status validate_depthwise(const Input &in, const Options &opt, std::string &err) {
    if (in.dw_stride == 0)
        return OK;
    if (in.dw_stride != 1 && in.dw_stride != 2) {
        err = "dw_stride must be 1 or 2 (got " + std::to_string(in.dw_stride) + ")";
        return E_ARG;
    }
    if (!in.dw_weights) {
        err = "dw_weights is NULL";
        return E_ARG;
    }
    if (in.dw_act < 0 || in.dw_act > 2) {
        err = "dw_act must be SPCONV_ACT_NONE, _RELU or _RELU6";
        return E_ARG;
    }
    if (in.storage != 0) {
        err = "the fused depthwise stage supports fp32 storage only";
        return E_UNSUPPORTED;
    }
    if (opt.kernel == 2) {
        err = "the fused depthwise stage needs the LDS-strip kernel (kernel = 2 was requested)";
        return E_UNSUPPORTED;
    }
    if (opt.pipe_sets || opt.regions) {
        err = "pipe_sets and regions select the pipelined kernel, which has no depthwise stage";
        return E_UNSUPPORTED;
    }
    for (int64_t i = 0; i < static_cast<int64_t>(in.cin) * 9; ++i) {
        if (!std::isfinite(in.dw_weights[i])) {
            err = "dw_weights[" + std::to_string(i / 9) + "][" + std::to_string(i % 9 / 3) + "][" +
                  std::to_string(i % 3) + "] is not finite";
            return E_FORMAT;
        }
    }
    for (int32_t c = 0; in.dw_bias && c < in.cin; ++c) {
        if (!std::isfinite(in.dw_bias[c])) {
            err = "dw_bias[" + std::to_string(c) + "] is not finite";
            return E_FORMAT;
        }
    }
    return OK;
}

// Input-channel blocks as the kernels' entries: block t of a row becomes kc
// entries (channels col_idx[t] .. + kc - 1, in order), each with the block's
// k output-channel values of that channel.  The per-row order stays ascending
// channel, so the result is the same as for the equivalent unblocked weight.
static void expand_input_blocks(const Input &in, std::vector<int32_t> &row_ptr, std::vector<int32_t> &col_idx,
                         std::vector<float> &values) {
    const int32_t k = in.block_rows, kc = in.block_cols, rows = in.cout / k;
    const int64_t nnzb = in.row_ptr[rows];
    row_ptr.resize(rows + 1);
    for (int32_t r = 0; r <= rows; ++r)
        row_ptr[r] = in.row_ptr[r] * kc;
    col_idx.resize(static_cast<size_t>(nnzb * kc));
    values.resize(static_cast<size_t>(nnzb * kc * k));
    for (int64_t t = 0; t < nnzb; ++t)
        for (int32_t j = 0; j < kc; ++j) {
            col_idx[t * kc + j] = in.col_idx[t] + j;
            for (int32_t i = 0; i < k; ++i)
                values[(t * kc + j) * k + i] = in.values[(t * k + i) * kc + j];
        }
}

Status build_plan(const Input &in_arg, const Options &opt, PackedPlan &p, std::string &err) {
    Status st = validate(in_arg, err);
    if (st != OK)
        return st;
    Input in = in_arg;
    std::vector<int32_t> xrow_ptr, xcol_idx;
    std::vector<float> xvalues;
    if (in.block_cols > 1) {
        expand_input_blocks(in_arg, xrow_ptr, xcol_idx, xvalues);
        in.row_ptr = xrow_ptr.data();
        in.col_idx = xcol_idx.data();
        in.values = xvalues.data();
        in.block_cols = 1;
    }
    if (opt.kernel < 0 || opt.kernel > 4) {
        err = "kernel must be 0 (automatic), 1 (strip), 2 (direct), 3 (register-indexed), 4 (lockstep) or 5 "
              "(channel-range passes)";
        return E_ARG;
    }
    if (opt.kernel == 4 && !outer_supported(in)) {
        err = "the lockstep kernel runs plans without a depthwise stage of 1 x 4 blocks with cin <= " +
              std::to_string(kOuterMaxCin32) + " or unstructured with cin <= " + std::to_string(kOuterMaxCin16);
        return E_UNSUPPORTED;
    }
    if (opt.kernel == 3 && (in.dw_stride || in.storage != 0)) {
        err = "the register-indexed kernel runs fp32 plans without a depthwise stage";
        return E_UNSUPPORTED;
    }
    if (opt.lane_cols < 0 || opt.lane_cols > 6) {
        err = "lane_cols must be 0 (automatic) or 1 .. 6";
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
    if (opt.pipe_sets < 0 || opt.pipe_sets > 2) {
        err = "pipe_sets must be 0, 1 or 2";
        return E_ARG;
    }
    if (opt.regions < 0 || opt.regions > kMaxRegions) {
        err = "regions must be in [0, " + std::to_string(kMaxRegions) + "]";
        return E_ARG;
    }
    st = validate_depthwise(in, opt, err);
    if (st != OK)
        return st;

    p = PackedPlan();
    p.cout = in.cout;
    p.cin = in.cin;
    p.k = in.block_rows;
    p.act = in.act;
    p.storage = in.storage;
    p.kc = in_arg.block_cols;
    Options gopt = opt;
    if (gopt.kernel == 3 || gopt.kernel == 4)
        gopt.kernel = 0;
    st = choose_geometry(in, gopt, p, err);
    if (st != OK)
        return st;
    if (in.dw_stride) {
        if (p.kernel != KERNEL_STRIP) {
            err = "the fused depthwise stage needs the LDS-strip kernel, and the strip of cin = " +
                  std::to_string(in.cin) + " channels does not fit in LDS";
            return E_UNSUPPORTED;
        }
        p.dw_stride = in.dw_stride;
        p.dw_act = in.dw_act;
        p.pipe_sets = 0;
        p.regions = 0;
        p.dw.assign(static_cast<size_t>(p.strip_rows) * kDwParams, 0.0f);
        for (int32_t c = 0; c < in.cin; ++c) {
            for (int32_t t = 0; t < 9; ++t)
                p.dw[static_cast<size_t>(c) * kDwParams + t] = in.dw_weights[static_cast<size_t>(c) * 9 + t];
            p.dw[static_cast<size_t>(c) * kDwParams + 9] = in.dw_bias ? in.dw_bias[c] : 0.0f;
        }
    }

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
    if (!in.dw_stride && in.storage == 0) {
        build_indexed(in, p.perm, p);
        p.use_indexed = opt.kernel == 3;
        p.rlane_cols = opt.lane_cols;
    }
    p.auto_kernel = opt.kernel == 0;
    if (outer_supported(in) && (opt.kernel == 0 || opt.kernel == 4)) {
        build_outer(in, p);
        p.use_outer = opt.kernel == 4;
    }

    // 2. bundles of NB consecutive entries in that order, each a whole number
    // of steps of 4 slots and at least one step long.  An entry is a row or,
    // for a row more than twice the median length (a heavy tail, which would
    // otherwise set the pace of its whole bundle and wavefront), one of its
    // two pieces: its even and its odd nonzeros, in two neighbouring lane
    // groups of one bundle, so both walk the channels at the same pace; the
    // second group's partial sums are added into the first's before the
    // epilogue.  Unstructured plans only, only with the length order, and not
    // in channel-range passes (each row summed in one ascending pass there).
    p.row_nnz.resize(rows);
    for (int32_t r = 0; r < rows; ++r)
        p.row_nnz[r] = len(r);
    struct Entry {
        int32_t row;    // -1: an empty lane group
        int32_t piece;  // -1 the whole row; 0 / 1 its even / odd nonzeros
    };
    auto elen = [&](const Entry &u) {
        return u.row < 0 ? 0 : u.piece < 0 ? len(u.row) : (len(u.row) + 1 - u.piece) / 2;
    };
    int32_t split_min = INT32_MAX;
    if (k == 1 && NB >= 2 && rows > 0 && opt.reorder && opt.split) {
        std::vector<int32_t> l(p.row_nnz);
        std::nth_element(l.begin(), l.begin() + rows / 2, l.end());
        split_min = std::max<int32_t>(kSplitMinNnz, 2 * l[rows / 2] + 1);
    }
    std::vector<Entry> ents;
    auto lay_out = [&](int32_t min_split) {
        ents.clear();
        p.split_rows = 0;
        std::vector<Entry> items;  // whole rows, and split rows as their first piece
        for (int32_t r : p.perm)
            items.push_back(Entry{r, len(r) >= min_split ? 0 : -1});
        std::stable_sort(items.begin(), items.end(), [&](const Entry &a, const Entry &b) { return elen(a) > elen(b); });
        for (const Entry &u : items) {
            if (u.piece < 0) {
                ents.push_back(u);
                continue;
            }
            if (ents.size() % 2)  // the two pieces take groups 2i and 2i + 1 of one bundle (NB is even)
                ents.push_back(Entry{-1, -1});
            ents.push_back(Entry{u.row, 0});
            ents.push_back(Entry{u.row, 1});
            ++p.split_rows;
        }
    };
    // split only where the longest row alone would take more than 1.5x the
    // average wavefront's steps of the unsplit layout (a nearly balanced plan
    // gains less than its extra entries and epilogue exchanges cost)
    if (split_min < INT32_MAX) {
        lay_out(INT32_MAX);
        int64_t steps0 = 0;
        for (int32_t b = 0; b < bundles_of(rows, NB); ++b) {
            int32_t l = 0;
            for (int32_t q = 0; q < NB; ++q) {
                const size_t at = static_cast<size_t>(b) * NB + q;
                if (at < ents.size())
                    l = std::max(l, elen(ents[at]));
            }
            steps0 += std::max<int32_t>(1, (l + kStepSlots - 1) / kStepSlots);
        }
        const int32_t w0 = opt.waves ? opt.waves : std::min<int32_t>(kMaxWaves, bundles_of(rows, NB));
        const int32_t longest = (len(p.perm[0]) + kStepSlots - 1) / kStepSlots;
        if (2 * static_cast<int64_t>(longest) * w0 <= 3 * steps0)
            split_min = INT32_MAX;
    }
    lay_out(split_min);
    if (p.split_rows) {
        // the bundle table (kept in LDS) grows with the extra entries: keep
        // the split only if it still fits
        const int64_t grow = table_bytes(bundles_of(static_cast<int32_t>(ents.size()), NB), NB, k) -
                             table_bytes(bundles_of(rows, NB), NB, k);
        if (p.lds_bytes + grow <= kMaxLdsBytes)
            p.lds_bytes += static_cast<int32_t>(grow);
        else
            lay_out(INT32_MAX);
    }
    const int32_t nb = bundles_of(static_cast<int32_t>(ents.size()), NB);
    ents.resize(static_cast<size_t>(nb) * NB, Entry{-1, -1});
    std::vector<int32_t> bsteps(nb, 0);
    for (int32_t b = 0; b < nb; ++b) {
        int32_t l = 0;
        for (int32_t q = 0; q < NB; ++q)
            l = std::max(l, elen(ents[static_cast<size_t>(b) * NB + q]));
        bsteps[b] = std::max<int32_t>(1, (l + kStepSlots - 1) / kStepSlots);
    }

    // 3. longest-processing-time-first assignment of bundles to waves
    // (as many as the unsplit layout would have: more wavefronts per
    // workgroup could cost resident workgroups)
    const int32_t waves = opt.waves ? opt.waves : std::min<int32_t>(kMaxWaves, bundles_of(rows, NB));
    p.waves = waves;
    if (p.dw_stride) {
        // the LDS left after the strip and the bundle table stages input
        // windows; a plan with at most 8 wavefronts keeps room for 2 (4: 3)
        // workgroups per CU, so one's depthwise phase overlaps another's 1x1
        p.stage_off = p.lds_bytes - kCtlBytes;
        const int32_t want = std::min<int32_t>(3, std::max<int32_t>(1, kMaxWaves / std::max(p.waves, 1)));
        for (int32_t o = want; o >= 1; --o) {
            const int64_t budget = (kMaxLdsBytes / o) & ~int64_t(255);
            const int64_t stage = (budget - kCtlBytes - p.stage_off) & ~int64_t(15);
            if (o == 1 || stage >= kMinStageBytes) {
                p.lds_bytes = static_cast<int32_t>(budget);
                p.stage_bytes = static_cast<int32_t>(stage);
                break;
            }
        }
    }
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
    const int32_t pad_channel = p.kernel == KERNEL_STRIP ? p.strip_rows : 0;
    p.idx.assign(static_cast<size_t>(total_steps * NB * kStepSlots), pad_channel * p.row_scale);
    p.val.assign(static_cast<size_t>(total_steps * NB * kStepSlots * k), 0.0f);
    p.wave_ptr.assign(waves + 1, 0);
    p.hdr.reserve(2 * static_cast<size_t>(nb));
    p.rows.reserve(static_cast<size_t>(NB) * nb);
    p.bundle_bias.reserve(static_cast<size_t>(NB) * nb * k);
    p.rank.reserve(nb);
    int64_t step = 0;   // first step of the next bundle
    int32_t bglob = 0;  // bundles packed so far
    for (int32_t w = 0; w < waves; ++w) {
        for (int32_t b : lists[w]) {
            p.hdr.push_back(static_cast<int32_t>(step));
            p.hdr.push_back(bsteps[b]);
            p.rank.push_back(rank_of[b]);
            for (int32_t q = 0; q < NB; ++q) {
                const Entry u = ents[static_cast<size_t>(b) * NB + q];
                const int32_t rb = u.row;
                p.rows.push_back(u.piece == 1 ? kRowPiece : rb);
                for (int32_t i = 0; i < k; ++i)
                    p.bundle_bias.push_back(rb >= 0 && u.piece != 1 && in.bias ? in.bias[rb * k + i] : 0.0f);
                if (rb < 0)
                    continue;
                const int32_t r0 = in.row_ptr[rb];
                const int32_t n = elen(u);
                for (int32_t t = 0; t < n; ++t) {
                    const int32_t s = u.piece < 0 ? t : 2 * t + u.piece;  // the row's nonzero in slot t
                    const int64_t e = ((step + t / kStepSlots) * NB + q) * kStepSlots + t % kStepSlots;
                    p.idx[e] = in.col_idx[r0 + s] * p.row_scale;
                    for (int32_t i = 0; i < k; ++i) {
                        float v = in.values[static_cast<int64_t>(r0 + s) * k + i];
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
        if (!lists[w].empty())
            ++p.busy_waves;
    }
    p.slots = total_steps * NB * kStepSlots;
    p.max_parts = 1;
    while (p.max_parts * 2 <= std::min<int32_t>(kMaxParts, nb))
        p.max_parts *= 2;

    // 5. interleaved streams for the pipelined strip kernel: two accumulator
    // sets when both fit in the automatic accumulator budget (a plan with a
    // depthwise stage runs the simple loop and needs none)
    if (p.kernel == KERNEL_STRIP && !p.dw_stride) {
        const int32_t acc = k * (p.cols_per_lane);
        const int32_t max_sets = 2 * acc <= kAutoAccumulators ? 2 : 1;
        if (opt.pipe_sets > max_sets) {
            err = "pipe_sets = 2 needs " + std::to_string(2 * acc) + " accumulators per lane (limit " +
                  std::to_string(kAutoAccumulators) + ")";
            return E_UNSUPPORTED;
        }
        p.pipe_sets = opt.pipe_sets ? opt.pipe_sets : max_sets;
        // automatic: about one part per kAutoRegionRows channels (measured on
        // MI355X: a part's refill is a workgroup-wide dependency, and narrow
        // strips run fastest in one or two parts, 512 channels in three)
        const int32_t auto_regions = std::max(1, std::min(kMaxRegions, (p.strip_rows + kAutoRegionRows - 1) / kAutoRegionRows));
        p.regions = std::min(opt.regions ? opt.regions : auto_regions, p.strip_rows / 4);
        p.region_rows = (p.strip_rows / 4 + p.regions - 1) / p.regions * 4;
        p.regions = (p.strip_rows + p.region_rows - 1) / p.region_rows;  // none left empty
        build_interleaved(p);
    }
    return OK;
}

// What lane group q of bundle b holds: a whole row, a piece of a split row
// (0: its even nonzeros, 1: its odd ones; the second piece's table entry is
// kRowPiece, after the first), or nothing; and how many real entries.
GroupRow group_row(const PackedPlan &p, int32_t b, int32_t q) {
    const int32_t NB = p.bundle_rows;
    const size_t at = static_cast<size_t>(b) * NB + q;
    const int32_t rb = p.rows[at];
    GroupRow gr{rb, -1, 0};
    if (rb == kRowPiece) {
        gr.row = q > 0 ? p.rows[at - 1] : -1;
        gr.piece = 1;
    } else if (rb >= 0 && q + 1 < NB && p.rows[at + 1] == kRowPiece) {
        gr.piece = 0;
    }
    if (gr.row >= 0 && gr.row < static_cast<int32_t>(p.row_nnz.size())) {
        const int32_t l = p.row_nnz[gr.row];
        gr.n = gr.piece < 0 ? l : (l + 1 - gr.piece) / 2;
    } else {
        gr.row = -1;
    }
    return gr;
}

void unpack_plan(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, int32_t *perm) {
    const int32_t k = p.k;
    const int32_t rows = p.cout / k;
    const int32_t NB = p.bundle_rows;
    std::vector<std::vector<int32_t>> cols(rows);
    std::vector<std::vector<float>> vals(rows);
    for (int32_t r = 0; r < rows; ++r) {
        cols[r].assign(p.row_nnz[r], -1);
        vals[r].assign(static_cast<size_t>(p.row_nnz[r]) * k, 0.0f);
    }
    // a lane group's real entries are the first ones of its sequence: the
    // whole row, or the even / odd nonzeros of a split row
    for (int32_t b = 0; b < p.nbundles(); ++b) {
        const int64_t s_first = p.hdr[2 * b];
        for (int32_t q = 0; q < NB; ++q) {
            const GroupRow gr = group_row(p, b, q);
            if (gr.row < 0)
                continue;
            for (int32_t t = 0; t < gr.n; ++t) {
                const int64_t e = ((s_first + t / kStepSlots) * NB + q) * kStepSlots + t % kStepSlots;
                const int32_t s = gr.piece < 0 ? t : 2 * t + gr.piece;
                cols[gr.row][s] = p.idx[e] / p.row_scale;
                for (int32_t i = 0; i < k; ++i)
                    vals[gr.row][static_cast<size_t>(s) * k + i] = p.val[e * k + i];
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

Status unpack_interleaved(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values,
                          std::string &err) {
    if (p.kernel != KERNEL_STRIP || p.pidx.size() != p.idx.size()) {
        err = "the plan has no interleaved streams (direct kernel or depthwise stage)";
        return E_FORMAT;
    }
    const int32_t k = p.k, NB = p.bundle_rows, S = p.pipe_sets;
    const int32_t rows = p.cout / k;
    std::vector<std::vector<int32_t>> cols(rows);
    std::vector<std::vector<float>> vals(rows);
    for (int32_t r = 0; r < rows; ++r) {
        cols[r].assign(p.row_nnz[r], -1);
        vals[r].assign(static_cast<size_t>(p.row_nnz[r]) * k, 0.0f);
    }
    auto bad = [&](const std::string &m) {
        err = m;
        return E_FORMAT;
    };
    for (int32_t w = 0; w < p.waves; ++w) {
        const int32_t b0 = p.wave_ptr[w], b1 = p.wave_ptr[w + 1];
        if (b0 == b1)
            continue;
        const int64_t ws0 = p.hdr[2 * b0];
        int64_t len = 0;
        for (int32_t b = b0; b < b1; ++b)
            len += p.hdr[2 * b + 1];
        // decode the events: first and last step allowed to read each region
        std::vector<int64_t> lo(kMaxRegions, INT64_MAX), hi(kMaxRegions, -1);
        for (int32_t i = 0; i < kMaxRegions; ++i) {
            const int32_t n = p.wave_ev[static_cast<size_t>(w) * kWaveEvents + i];
            const int32_t r = p.wave_ev[static_cast<size_t>(w) * kWaveEvents + kMaxRegions + i];
            if (n != INT32_MAX)
                lo[n & 15] = n >> 4;
            if (r != INT32_MAX)
                hi[r & 15] = r >> 4;
        }
        std::vector<int32_t> bset(S), cnt(S, 0);
        for (int32_t i = 0; i < S; ++i)
            bset[i] = b0 + i;
        for (int64_t i = 0; i < len; ++i) {
            const uint32_t bits = p.psel[p.sel_ptr[w] + i / kSelSteps] >> (2 * (i % kSelSteps)) & 3u;
            const int32_t set = static_cast<int32_t>(bits & 1u);
            if (set >= S)
                return bad("selector names a set the plan does not have");
            const int32_t b = bset[set];
            if (b >= b1 || cnt[set] >= p.hdr[2 * b + 1])
                return bad("selector runs past a wavefront's bundles");
            const int64_t step = ws0 + i;
            for (int32_t q = 0; q < NB; ++q) {
                const GroupRow gr = group_row(p, b, q);
                const int32_t rb = gr.row;
                for (int32_t u = 0; u < kStepSlots; ++u) {
                    const int64_t e = (step * NB + q) * kStepSlots + u;
                    const int32_t c = p.pidx[e] / p.row_scale;
                    const int32_t t = cnt[set] * kStepSlots + u;
                    if (rb < 0 || t >= gr.n) {
                        if (c != p.strip_rows)
                            return bad("a padding slot reads a strip channel");
                        for (int32_t j = 0; j < k; ++j)
                            if (p.pval[e * k + j] != 0.0f)
                                return bad("a padding slot has a nonzero weight");
                        continue;
                    }
                    const int32_t r = c / p.region_rows;
                    if (c < 0 || c >= p.strip_rows || i < lo[r] || i > hi[r])
                        return bad("a step reads a strip part outside its need / release events");
                    const int32_t sl = gr.piece < 0 ? t : 2 * t + gr.piece;
                    cols[rb][sl] = c;
                    for (int32_t j = 0; j < k; ++j)
                        vals[rb][static_cast<size_t>(sl) * k + j] = p.pval[e * k + j];
                }
            }
            ++cnt[set];
            const bool last = cnt[set] == p.hdr[2 * b + 1];
            if (last != ((bits & 2u) != 0))
                return bad("a last-step bit disagrees with the bundle length");
            if (last) {
                bset[set] += S;
                cnt[set] = 0;
            }
        }
        for (int32_t i = 0; i < S; ++i)
            if (bset[i] < b1)
                return bad("a wavefront's stream ends before its bundles do");
    }
    for (int32_t r = 0; r < rows; ++r)
        if (std::find(cols[r].begin(), cols[r].end(), -1) != cols[r].end())
            return bad("row " + std::to_string(r) + " has entries no stream holds");
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
    return OK;
}

}  // namespace spconv

namespace spconv {

// Register-indexed kernel: slots, records, row pairs (planner.hpp).
void build_indexed(const Input &in, const std::vector<int32_t> &order, PackedPlan &p) {
    const int32_t k = in.block_rows;
    const int32_t rows = in.cout / k;           // block rows
    const int32_t cap = kSlotRows / k;          // block rows per slot
    const int32_t S = (rows + cap - 1) / cap;
    const int32_t G = (S + kSlotsPerGroup - 1) / kSlotsPerGroup;
    const int32_t W = (S + G - 1) / G;
    const int32_t nch = (in.cin + kChunk - 1) / kChunk;
    const int32_t P = rec_slots(k);
    auto len = [&](int32_t r) { return in.row_ptr[r + 1] - in.row_ptr[r]; };
    auto weight = [&](int64_t t, int32_t i) {
        float v = in.values[t * k + i];
        if (in.storage == 1)
            v = half_to_float(float_to_half_rne(v));
        return v;
    };
    p.rslots = S;
    p.rgroups = G;
    p.rwaves = W;
    p.rnch = nch;

    // 1. slots: heaviest block rows first, each to the least loaded slot with room
    std::vector<std::vector<int32_t>> members(S);
    std::vector<int64_t> load(S, 0);
    for (int32_t rb : order) {
        int32_t best = -1;
        for (int32_t s = 0; s < S; ++s)
            if (static_cast<int32_t>(members[s].size()) < cap && (best < 0 || load[s] < load[best]))
                best = s;
        members[best].push_back(rb);
        load[best] += len(rb);
    }
    p.rslot_rows.assign(static_cast<size_t>(S) * kSlotRows, -1);
    p.rslot_bias.assign(static_cast<size_t>(S) * kSlotRows, 0.0f);
    for (int32_t s = 0; s < S; ++s) {
        std::sort(members[s].begin(), members[s].end());
        for (int32_t b = 0; b < static_cast<int32_t>(members[s].size()); ++b)
            for (int32_t i = 0; i < k; ++i) {
                const int32_t r = members[s][b] * k + i;
                p.rslot_rows[static_cast<size_t>(s) * kSlotRows + b * k + i] = r;
                p.rslot_bias[static_cast<size_t>(s) * kSlotRows + b * k + i] = in.bias ? in.bias[r] : 0.0f;
            }
    }

    // 2. records: per slot, per channel ascending, groups of at most P blocks
    p.rrec.clear();
    p.rslot_batch.assign(S, 0);
    p.rslot_chunk.assign(static_cast<size_t>(S) * (nch + 1), 0);
    p.rslot_nrec.assign(static_cast<size_t>(S) * nch, 0);
    const int32_t batch_words = kRecWords * kBatchRecs;
    const int32_t F = flag_word(k);
    for (int32_t s = 0; s < S; ++s) {
        const int64_t first_batch = static_cast<int64_t>(p.rrec.size()) / batch_words;
        p.rslot_batch[s] = static_cast<int32_t>(first_batch);
        // (channel, slot position, stored-block index) of every block of the slot
        struct Ent {
            int32_t c, pos;
            int64_t t;
        };
        std::vector<Ent> ents;
        for (int32_t b = 0; b < static_cast<int32_t>(members[s].size()); ++b) {
            const int32_t rb = members[s][b];
            for (int32_t t = in.row_ptr[rb]; t < in.row_ptr[rb + 1]; ++t)
                ents.push_back({in.col_idx[t], b, t});
        }
        std::stable_sort(ents.begin(), ents.end(), [](const Ent &a, const Ent &b) {
            return a.c != b.c ? a.c < b.c : a.pos < b.pos;
        });
        size_t e = 0;
        for (int32_t q = 0; q < nch; ++q) {
            const size_t chunk_start = p.rrec.size();
            p.rslot_chunk[static_cast<size_t>(s) * (nch + 1) + q] =
                static_cast<int32_t>(static_cast<int64_t>(chunk_start) / batch_words - first_batch);
            int32_t nrec = 0;
            while (e < ents.size() && ents[e].c < (q + 1) * kChunk) {
                const int32_t c = ents[e].c;
                size_t e1 = e;
                while (e1 < ents.size() && ents[e1].c == c)
                    ++e1;
                for (size_t g = e; g < e1; g += P) {
                    const int32_t n = static_cast<int32_t>(std::min<size_t>(P, e1 - g));
                    uint32_t w[kRecWords] = {0, 0, 0, 0, 0, 0, 0, 0};
                    w[0] = static_cast<uint32_t>((c % kRing) * kRingRowBytes);
                    for (int32_t j = 0; j < n; ++j) {
                        const uint32_t row = static_cast<uint32_t>(ents[g + j].pos * k);
                        w[1 + j] = row;
                        for (int32_t i = 0; i < k; ++i) {
                            const float v = weight(ents[g + j].t, i);
                            std::memcpy(&w[4 + j * k + i], &v, 4);
                        }
                    }
                    if (n > 1)
                        w[1] |= 1u << 8;
                    if (n > 2)
                        w[1] |= 1u << 9;
                    p.rrec.insert(p.rrec.end(), w, w + kRecWords);
                    ++nrec;
                }
                e = e1;
            }
            p.rslot_nrec[static_cast<size_t>(s) * nch + q] = nrec;
            // pad to whole batches, at least one: weight-0 records on the chunk's first channel
            const int32_t padded = std::max<int32_t>(kBatchRecs, (nrec + kBatchRecs - 1) / kBatchRecs * kBatchRecs);
            for (int32_t r = nrec; r < padded; ++r) {
                uint32_t w[kRecWords] = {static_cast<uint32_t>(((q * kChunk) % kRing) * kRingRowBytes), 0, 0, 0, 0, 0, 0, 0};
                p.rrec.insert(p.rrec.end(), w, w + kRecWords);
            }
            p.rrec[p.rrec.size() - batch_words + F] |= kLastOfChunk;
        }
        p.rrec[p.rrec.size() - batch_words + F] |= kLastOfStream;
        const int64_t total = static_cast<int64_t>(p.rrec.size()) / batch_words - first_batch;
        p.rslot_chunk[static_cast<size_t>(s) * (nch + 1) + nch] = static_cast<int32_t>(total);
    }
    p.rrec.insert(p.rrec.end(), static_cast<size_t>(2 * batch_words), 0u);

    // 3. row pairs
    p.rrow_bias.assign(in.cout, 0.0f);
    if (in.bias)
        std::copy(in.bias, in.bias + in.cout, p.rrow_bias.begin());
    const int32_t npairs = (in.cout + 1) / 2;
    p.rpair_ptr.assign(npairs + 1, 0);
    p.rpair_ent.clear();
    for (int32_t j = 0; j < npairs; ++j) {
        // the blocks of output channels 2j and 2j + 1 (block row r / k, element r % k)
        int32_t ra = 2 * j, rbb = 2 * j + 1;
        std::vector<std::pair<int32_t, int32_t>> lst;  // (channel, which) for stored (row, channel)
        struct W2 {
            float a = 0.0f, b = 0.0f;
            uint32_t mask = 0;
        };
        std::vector<int32_t> chans;
        std::vector<W2> ws;
        auto add_row = [&](int32_t r, int32_t which) {
            if (r >= in.cout)
                return;
            const int32_t rb = r / k, i = r % k;
            for (int32_t t = in.row_ptr[rb]; t < in.row_ptr[rb + 1]; ++t)
                lst.push_back({in.col_idx[t], which});
            (void)i;
        };
        add_row(ra, 0);
        add_row(rbb, 1);
        std::sort(lst.begin(), lst.end());
        for (size_t u = 0; u < lst.size(); ++u) {
            const int32_t c = lst[u].first;
            if (chans.empty() || chans.back() != c) {
                chans.push_back(c);
                ws.push_back(W2());
            }
            const int32_t r = lst[u].second ? rbb : ra;
            const int32_t rb = r / k, i = r % k;
            const int32_t *b0 = in.col_idx + in.row_ptr[rb];
            const int32_t *b1 = in.col_idx + in.row_ptr[rb + 1];
            const int64_t t = std::lower_bound(b0, b1, c) - in.col_idx;
            const float v = weight(t, i);
            if (lst[u].second) {
                ws.back().b = v;
                ws.back().mask |= 2u;
            } else {
                ws.back().a = v;
                ws.back().mask |= 1u;
            }
        }
        for (size_t u = 0; u < chans.size(); ++u) {
            uint32_t w[4];
            w[0] = static_cast<uint32_t>(chans[u]) | (ws[u].mask << 24);
            std::memcpy(&w[1], &ws[u].a, 4);
            std::memcpy(&w[2], &ws[u].b, 4);
            w[3] = 0;
            p.rpair_ent.insert(p.rpair_ent.end(), w, w + 4);
        }
        p.rpair_ptr[j + 1] = static_cast<int32_t>(p.rpair_ent.size() / 4);
    }
}

Status unpack_indexed(const PackedPlan &p, bool from_pairs, int32_t *row_ptr, int32_t *col_idx, float *values,
                      std::string &err) {
    if (p.rslots == 0) {
        err = "the plan has no register-indexed streams";
        return E_FORMAT;
    }
    const int32_t k = p.k;
    const int32_t rows = p.cout / k;
    std::vector<std::vector<int32_t>> cols(rows);
    std::vector<std::vector<float>> vals(rows);
    auto bad = [&](const std::string &m) {
        err = m;
        return E_FORMAT;
    };
    auto fl = [](uint32_t u) {
        float v;
        std::memcpy(&v, &u, 4);
        return v;
    };
    const int32_t nch = p.rnch;
    const int32_t P = rec_slots(k);
    if (!from_pairs) {
        // (block row, element) -> its column and value lists are filled per block row;
        // per-row element values are collected block-major
        std::vector<std::vector<int32_t>> bc(rows);
        std::vector<std::vector<std::vector<float>>> bv(rows);
        for (int32_t s = 0; s < p.rslots; ++s) {
            const int64_t base = static_cast<int64_t>(p.rslot_batch[s]) * kBatchRecs;  // first record
            const int32_t *ch = p.rslot_chunk.data() + static_cast<size_t>(s) * (nch + 1);
            const int32_t *nr = p.rslot_nrec.data() + static_cast<size_t>(s) * nch;
            const int32_t F = flag_word(k);
            int32_t prev_c = -1;
            for (int32_t q = 0; q < nch; ++q) {
                const int32_t b0 = ch[q], b1 = ch[q + 1];
                const int64_t nrec = nr[q];
                if (b1 <= b0 || nrec < 0 || (b1 - b0) != std::max<int64_t>(1, (nrec + kBatchRecs - 1) / kBatchRecs))
                    return bad("chunk table out of order");
                // flags: only the chunk's last batch ends it, only the stream's last ends the stream
                for (int32_t bb = b0; bb < b1; ++bb) {
                    const uint32_t f = p.rrec[(base + static_cast<int64_t>(bb) * kBatchRecs) * kRecWords + F];
                    const uint32_t want =
                        (bb == b1 - 1 ? kLastOfChunk : 0u) | (q == nch - 1 && bb == b1 - 1 ? kLastOfStream : 0u);
                    if ((f & 3u) != want)
                        return bad("batch flags do not match the chunk table");
                }
                for (int64_t r = 0; r < nrec; ++r) {
                    const uint32_t *w = p.rrec.data() + (base + static_cast<int64_t>(b0) * kBatchRecs + r) * kRecWords;
                    const int32_t n = 1 + ((w[1] >> 8) & 1) + ((w[1] >> 9) & 1);
                    if (n > P)
                        return bad("record holds more blocks than its kind allows");
                    // the channel: the ring row plus the chunk's ring base
                    const int32_t c =
                        (q * kChunk) / kRing * kRing + static_cast<int32_t>(w[0] / static_cast<uint32_t>(kRingRowBytes));
                    if (w[0] % kRingRowBytes || w[0] >= static_cast<uint32_t>(kRing * kRingRowBytes) || c < q * kChunk ||
                        c >= (q + 1) * kChunk || c >= p.cin)
                        return bad("record channel outside its chunk");
                    if (c < prev_c)
                        return bad("records do not ascend by channel");
                    prev_c = c;
                    for (int32_t j = 0; j < n; ++j) {
                        const uint32_t row = w[1 + j] & 0xffu;
                        if (row % k || static_cast<int32_t>(row) >= kSlotRows)
                            return bad("slot row out of range");
                        const int32_t orow = p.rslot_rows[static_cast<size_t>(s) * kSlotRows + row];
                        if (orow < 0 || orow % k)
                            return bad("record names an unused slot row");
                        const int32_t rb = orow / k;
                        bc[rb].push_back(c);
                        std::vector<float> v(k);
                        for (int32_t i = 0; i < k; ++i)
                            v[i] = fl(w[4 + j * k + i]);
                        bv[rb].push_back(v);
                    }
                }
            }
        }
        for (int32_t rb = 0; rb < rows; ++rb) {
            std::vector<size_t> idx(bc[rb].size());
            std::iota(idx.begin(), idx.end(), 0);
            std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) { return bc[rb][a] < bc[rb][b]; });
            for (size_t u : idx) {
                cols[rb].push_back(bc[rb][u]);
                for (int32_t i = 0; i < k; ++i)
                    vals[rb].push_back(bv[rb][u][i]);
            }
        }
    } else {
        // per output channel, its (channel, value) list; blocks are rebuilt per block row
        std::vector<std::vector<std::pair<int32_t, float>>> orow(p.cout);
        const int32_t npairs = static_cast<int32_t>(p.rpair_ptr.size()) - 1;
        for (int32_t j = 0; j < npairs; ++j) {
            int32_t prev = -1;
            for (int32_t u = p.rpair_ptr[j]; u < p.rpair_ptr[j + 1]; ++u) {
                const uint32_t *w = p.rpair_ent.data() + static_cast<size_t>(u) * 4;
                const int32_t c = static_cast<int32_t>(w[0] & 0xffffffu);
                const uint32_t mask = w[0] >> 24;
                if (c <= prev || c >= p.cin || mask == 0 || mask > 3)
                    return bad("pair entries malformed");
                prev = c;
                if (mask & 1u)
                    orow[2 * j].push_back({c, fl(w[1])});
                if (mask & 2u) {
                    if (2 * j + 1 >= p.cout)
                        return bad("pair entry for a row past cout");
                    orow[2 * j + 1].push_back({c, fl(w[2])});
                }
            }
        }
        for (int32_t rb = 0; rb < rows; ++rb) {
            const auto &lead = orow[rb * k];
            for (int32_t i = 1; i < k; ++i)
                if (orow[rb * k + i].size() != lead.size())
                    return bad("rows of one block differ in their channels");
            for (size_t u = 0; u < lead.size(); ++u) {
                cols[rb].push_back(lead[u].first);
                for (int32_t i = 0; i < k; ++i) {
                    if (orow[rb * k + i][u].first != lead[u].first)
                        return bad("rows of one block differ in their channels");
                    vals[rb].push_back(orow[rb * k + i][u].second);
                }
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
    return OK;
}

}  // namespace spconv

namespace spconv {

// Lockstep kernel: group sets, records, wave lists (planner.hpp).
bool outer_supported(const Input &in) {
    if (in.dw_stride != 0 || in.cin < 1)
        return false;
    return (in.block_rows == 4 && in.cin <= kOuterMaxCin32) ||
           (in.block_rows == 1 && in.storage == 0 && in.cin <= kOuterMaxCin16);
}

void build_outer(const Input &in, PackedPlan &p) {
    const int32_t k = in.block_rows;
    const int32_t rows = in.cout / k;
    auto len = [&](int32_t r) { return in.row_ptr[r + 1] - in.row_ptr[r]; };
    std::vector<int32_t> order(rows);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return len(a) > len(b); });
    p.omode = k == 4 ? 0 : 1;
    p.otw = p.omode == 0 || in.cin <= kOuterMaxCin32 ? 32 : 16;
    p.ogroups = 256 / p.otw;
    const int32_t G = p.ogroups;
    const int32_t row_bytes = 4 * p.otw;
    const int32_t per_copy = 1024 / row_bytes;  // rows one 1 KB copy instruction moves
    const int32_t kw = k == 4 ? 4 : 1;          // weight slots per group
    const int32_t slots = G * kw;
    const int32_t O = (rows + G - 1) / G;
    p.oocts = O;
    p.ozrow = (in.cin + per_copy - 1) / per_copy * per_copy;
    const uint32_t zoff = static_cast<uint32_t>(p.ozrow * row_bytes);
    p.orec.clear();
    p.ooff.clear();
    p.ooct_tab.assign(static_cast<size_t>(O) * kOctWords, 0);
    std::vector<int64_t> steps(O);
    int32_t quads = 0;
    for (int32_t o = 0; o < O; ++o) {
        int32_t l = 0;
        for (int32_t g = 0; g < G && o * G + g < rows; ++g)
            l = std::max(l, len(order[o * G + g]));
        const int32_t nq = std::max<int32_t>(1, (l + kOuterQuadSteps - 1) / kOuterQuadSteps);
        steps[o] = int64_t(kOuterQuadSteps) * nq;
        int32_t *tab = &p.ooct_tab[static_cast<size_t>(o) * kOctWords];
        tab[0] = quads;
        tab[1] = nq;
        quads += nq;
        for (int32_t g = 0; g < G; ++g)
            tab[2 + g] = o * G + g < rows ? order[o * G + g] : -1;
        for (int32_t j = 0; j < nq; ++j) {
            for (int32_t u = 0; u < slots; ++u) {
                const int32_t g = u / kw, t = u % kw, rb = tab[2 + g];
                for (int32_t h = 0; h < kOuterQuadSteps; ++h) {
                    const int32_t s = kOuterQuadSteps * j + h;
                    uint32_t w = 0;
                    if (rb >= 0 && s < len(rb)) {
                        float v = in.values[(static_cast<int64_t>(in.row_ptr[rb]) + s) * k + t];
                        if (in.storage == 1)
                            v = half_to_float(float_to_half_rne(v));
                        std::memcpy(&w, &v, 4);
                    }
                    p.orec.push_back(w);
                }
            }
            for (int32_t g = 0; g < G; ++g) {
                const int32_t rb = tab[2 + g];
                for (int32_t h = 0; h < kOuterQuadSteps; ++h) {
                    const int32_t s = kOuterQuadSteps * j + h;
                    p.ooff.push_back(rb >= 0 && s < len(rb)
                                         ? static_cast<uint32_t>(in.col_idx[in.row_ptr[rb] + s] * row_bytes)
                                         : zoff);
                }
            }
        }
    }
    p.orec.insert(p.orec.end(), static_cast<size_t>(kOuterAhead) * slots * 4, 0u);
    p.ooff.insert(p.ooff.end(), static_cast<size_t>(kOuterAhead) * G * 4, zoff);

    // wave lists: even tiles, then odd tiles continuing from the even loads
    const int32_t W = std::min<int32_t>(kMaxWaves, O);
    p.owaves = W;
    std::vector<int32_t> by_len(O);
    std::iota(by_len.begin(), by_len.end(), 0);
    std::stable_sort(by_len.begin(), by_len.end(), [&](int32_t a, int32_t b) { return steps[a] > steps[b]; });
    std::vector<int64_t> load(W, 0);
    std::vector<std::vector<int32_t>> lists(2 * W);
    for (int32_t q = 0; q < 2; ++q)
        for (int32_t o : by_len) {
            int32_t best = 0;
            for (int32_t w = 1; w < W; ++w)
                if (load[w] < load[best])
                    best = w;
            lists[q * W + best].push_back(o);
            load[best] += steps[o];
        }
    p.owave_ptr.assign(2 * W + 1, 0);
    p.owave_oct.clear();
    for (int32_t i = 0; i < 2 * W; ++i) {
        p.owave_ptr[i] = static_cast<int32_t>(p.owave_oct.size());
        p.owave_oct.insert(p.owave_oct.end(), lists[i].begin(), lists[i].end());
    }
    p.owave_ptr[2 * W] = static_cast<int32_t>(p.owave_oct.size());
    if (p.rrow_bias.size() != static_cast<size_t>(in.cout)) {
        p.rrow_bias.assign(in.cout, 0.0f);
        if (in.bias)
            std::copy(in.bias, in.bias + in.cout, p.rrow_bias.begin());
    }
}

Status unpack_outer(const PackedPlan &p, int32_t *row_ptr, int32_t *col_idx, float *values, std::string &err) {
    if (p.oocts == 0) {
        err = "the plan has no lockstep-kernel records";
        return E_FORMAT;
    }
    const int32_t k = p.k, rows = p.cout / k, O = p.oocts, W = p.owaves, G = p.ogroups;
    const int32_t kw = k == 4 ? 4 : 1, slots = G * kw;
    const int32_t row_bytes = 4 * p.otw, per_copy = 1024 / row_bytes;
    const uint32_t zoff = static_cast<uint32_t>(p.ozrow * row_bytes);
    if ((k != 1 && k != 4) || (p.omode != (k == 4 ? 0 : 1)) || (p.otw != 32 && p.otw != 16) ||
        G != 256 / p.otw || G + 2 > kOctWords || p.ozrow != (p.cin + per_copy - 1) / per_copy * per_copy ||
        static_cast<int32_t>(p.ooct_tab.size()) != O * kOctWords ||
        static_cast<int32_t>(p.owave_ptr.size()) != 2 * W + 1) {
        err = "lockstep-kernel geometry or tables are inconsistent";
        return E_FORMAT;
    }
    // every set exactly once per tile parity
    for (int32_t q = 0; q < 2; ++q) {
        std::vector<int32_t> seen(O, 0);
        for (int32_t i = p.owave_ptr[q * W]; i < p.owave_ptr[q * W + W]; ++i) {
            const int32_t o = p.owave_oct[i];
            if (o < 0 || o >= O || seen[o]++) {
                err = "wave lists do not cover every set once per tile parity";
                return E_FORMAT;
            }
        }
        if (std::count(seen.begin(), seen.end(), 1) != O) {
            err = "wave lists miss a set";
            return E_FORMAT;
        }
    }
    struct Blk {
        int32_t c;
        float w[4];
    };
    std::vector<std::vector<Blk>> got(rows);
    std::vector<int32_t> owner(rows, 0);
    int64_t next_quad = 0;
    for (int32_t o = 0; o < O; ++o) {
        const int32_t *tab = &p.ooct_tab[static_cast<size_t>(o) * kOctWords];
        const int64_t q0 = tab[0], nq = tab[1];
        if (q0 != next_quad || nq < 1 ||
            (q0 + nq + kOuterAhead) * slots * 4 > static_cast<int64_t>(p.orec.size()) ||
            (q0 + nq + kOuterAhead) * G * 4 > static_cast<int64_t>(p.ooff.size())) {
            err = "set " + std::to_string(o) + ": records out of order or out of range";
            return E_FORMAT;
        }
        next_quad = q0 + nq;
        for (int32_t g = 0; g < G; ++g) {
            const int32_t rb = tab[2 + g];
            if (rb < -1 || rb >= rows || (rb >= 0 && owner[rb]++)) {
                err = "set " + std::to_string(o) + ": bad or repeated block row";
                return E_FORMAT;
            }
            bool padding = rb < 0;
            int32_t last_c = -1;
            for (int64_t s = 0; s < kOuterQuadSteps * nq; ++s) {
                const int64_t j = q0 + s / kOuterQuadSteps, h = s % kOuterQuadSteps;
                Blk b{};
                for (int32_t t = 0; t < kw; ++t)
                    std::memcpy(&b.w[t], &p.orec[static_cast<size_t>((j * slots + kw * g + t) * 4 + h)], 4);
                const uint32_t off = p.ooff[static_cast<size_t>((j * G + g) * 4 + h)];
                if (off == zoff) {
                    for (int32_t t = 0; t < kw; ++t)
                        if (b.w[t] != 0.0f) {
                            err = "set " + std::to_string(o) + ": padding step with a nonzero weight";
                            return E_FORMAT;
                        }
                    padding = true;
                    continue;
                }
                if (padding || off % row_bytes || static_cast<int32_t>(off / row_bytes) >= p.cin ||
                    static_cast<int32_t>(off / row_bytes) <= last_c) {
                    err = "set " + std::to_string(o) + ": block after padding, bad offset or channels not ascending";
                    return E_FORMAT;
                }
                b.c = static_cast<int32_t>(off / row_bytes);
                last_c = b.c;
                got[rb].push_back(b);
            }
        }
    }
    if (static_cast<int64_t>(p.orec.size()) != (next_quad + kOuterAhead) * slots * 4 ||
        static_cast<int64_t>(p.ooff.size()) != (next_quad + kOuterAhead) * G * 4) {
        err = "record arrays' lengths do not match the sets";
        return E_FORMAT;
    }
    for (int32_t rb = 0; rb < rows; ++rb)
        if (!owner[rb]) {
            err = "block row " + std::to_string(rb) + " is in no set";
            return E_FORMAT;
        }
    int64_t nz = 0;
    for (int32_t rb = 0; rb < rows; ++rb) {
        if (row_ptr)
            row_ptr[rb] = static_cast<int32_t>(nz);
        for (const Blk &b : got[rb]) {
            if (col_idx)
                col_idx[nz] = b.c;
            if (values)
                for (int32_t t = 0; t < kw; ++t)
                    values[nz * kw + t] = b.w[t];
            ++nz;
        }
    }
    if (row_ptr)
        row_ptr[rows] = static_cast<int32_t>(nz);
    return OK;
}

}  // namespace spconv
