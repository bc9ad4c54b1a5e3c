// plan.cpp -- host-only planning for the swap engine: layer validation,
// prepacking into the device layout, lowering of user blocks to slabs under
// the pair constraint, two-ended arena placement, activation-slot placement
// and the pinned image.  No device calls.
//
// Paper correspondence: blocks of one or more layers run one by one
// (Sec. 3, "Basic Idea"); two consecutive blocks are resident together
// (m = 2 parallel blocks), which gives the constraint s_i + s_{i+1} <= b
// (Sec. 6.2.2, Eq. 3) and the block count n = ceil(m s / b); the skeleton
// (Sec. 5.2) becomes the piece table: for every parameter tensor an offset
// into its slab, so that assembly is pointer arithmetic.
#include <algorithm>
#include <cstring>

#include "engine.h"

namespace sn {

static bool set_err(std::string &err, const std::string &m) {
    err = m;
    return false;
}

// ---------------------------------------------------------------------------
// Validation and shape inference
// ---------------------------------------------------------------------------
static bool same_shape(const Slot &a, const Slot &b) {
    return a.h == b.h && a.w == b.w && a.c == b.c && a.cp == b.cp && a.rows == b.rows &&
           a.elem == b.elem;
}

static int define_slot(std::vector<Slot> &slots, int id, const Slot &shape, int li,
                       std::string &err) {
    if (id < 0 || id >= (int)slots.size())
        return set_err(err, "layer " + std::to_string(li) + ": dst slot out of range"), SN_E_INVALID;
    Slot &s = slots[id];
    if (s.used) {
        if (!same_shape(s, shape))
            return set_err(err, "layer " + std::to_string(li) + ": slot " + std::to_string(id) +
                                    " rewritten with a different shape"),
                   SN_E_INVALID;
    } else {
        int first = s.first;
        s = shape;
        s.used = true;
        s.first = first;
    }
    s.first = std::min(s.first, li);
    s.last = std::max(s.last, li);
    return SN_OK;
}

static int use_slot(std::vector<Slot> &slots, int id, int li, std::string &err, const Slot **out) {
    if (id < 0 || id >= (int)slots.size() || !slots[id].used)
        return set_err(err, "layer " + std::to_string(li) + ": reads slot " + std::to_string(id) +
                                " before any layer wrote it"),
               SN_E_INVALID;
    slots[id].last = std::max(slots[id].last, li);
    *out = &slots[id];
    return SN_OK;
}

static Slot image_slot(int h, int w, int c) {
    Slot s;
    s.h = h;
    s.w = w;
    s.c = c;
    s.cp = round8(c);
    s.rows = h * w;
    s.elem = 2;
    return s;
}

static Slot token_slot(int rows, int c, int elem) {
    Slot s;
    s.h = rows;
    s.w = 1;
    s.c = c;
    s.cp = c;
    s.rows = rows;
    s.elem = elem;
    return s;
}

static const int kMaxSlots = 4096;

// Validate layers [from, end) (appended by the latest sn_add_block), derive
// shapes and weight geometry.  `slots` carries state across calls.
int validate_layers(std::vector<Layer> &layers, int from, std::vector<Slot> &slots,
                    std::string &err) {
    if ((int)slots.size() < kMaxSlots) slots.resize(kMaxSlots);
    const bool token = !layers.empty() && layers[0].d.op == SN_OP_EMBED;
    int max_tokens = token ? layers[0].d.max_tokens : 0;
    for (int li = from; li < (int)layers.size(); ++li) {
        Layer &L = layers[li];
        const sn_layer &d = L.d;
        L.token = token;
        const std::string at = "layer " + std::to_string(li) + ": ";
        if (d.dst < 0 || d.dst >= kMaxSlots) return set_err(err, at + "bad dst slot"), SN_E_INVALID;
        if (d.res >= kMaxSlots || d.src >= kMaxSlots)
            return set_err(err, at + "slot id out of range"), SN_E_INVALID;
        if (d.w_bytes < 0 || d.b_bytes < 0 || d.w_off < 0 || d.b_off < 0)
            return set_err(err, at + "negative offset or size"), SN_E_INVALID;
        if (d.c_in <= 0 || d.c_out <= 0) return set_err(err, at + "channels must be > 0"), SN_E_INVALID;
        if (li > 0 && d.op == SN_OP_EMBED)
            return set_err(err, at + "embedding must be the first layer"), SN_E_INVALID;
        if (token && (d.op == SN_OP_CONV2D || d.op == SN_OP_MAXPOOL || d.op == SN_OP_GAVGPOOL ||
                      d.op == SN_OP_UPSAMPLE_BILINEAR))
            return set_err(err, at + "image op in a token network"), SN_E_UNSUPPORTED;
        if (!token && (d.op == SN_OP_RMSNORM || d.op == SN_OP_ATTENTION))
            return set_err(err, at + "token op in an image network"), SN_E_UNSUPPORTED;

        // network input: the first layer's src
        if (li == 0 && !token) {
            if (d.src < 0) return set_err(err, at + "bad src slot"), SN_E_INVALID;
            if (d.h_in <= 0 || d.w_in <= 0) return set_err(err, at + "bad input size"), SN_E_INVALID;
            Slot in = image_slot(d.h_in, d.w_in, d.c_in);
            if (d.op == SN_OP_LINEAR && !(d.flags & SN_FLAG_FLATTEN_CHW)) in = image_slot(1, 1, d.c_in);
            int rc = define_slot(slots, d.src, in, -1, err);
            if (rc) return rc;
        }
        const Slot *src = nullptr;
        if (d.op != SN_OP_EMBED) {
            int rc = use_slot(slots, d.src, li, err, &src);
            if (rc) return rc;
        }
        Slot out;
        switch (d.op) {
        case SN_OP_CONV2D: {
            if (d.k <= 0 || d.stride <= 0 || d.pad < 0 || d.dilation <= 0)
                return set_err(err, at + "bad conv geometry"), SN_E_INVALID;
            if (src->h != d.h_in || src->w != d.w_in || src->c != d.c_in)
                return set_err(err, at + "input slot shape does not match h_in/w_in/c_in"), SN_E_INVALID;
            int ho = (d.h_in + 2 * d.pad - d.dilation * (d.k - 1) - 1) / d.stride + 1;
            int wo = (d.w_in + 2 * d.pad - d.dilation * (d.k - 1) - 1) / d.stride + 1;
            if (ho <= 0 || wo <= 0) return set_err(err, at + "empty output"), SN_E_INVALID;
            L.out_h = ho;
            L.out_w = wo;
            L.cin_p = src->cp;
            L.K = d.k * d.k * L.cin_p;
            L.units = d.c_out;
            L.w_unit_bytes = (int64_t)L.K * 2;
            if (d.w_bytes != (int64_t)d.c_out * d.c_in * d.k * d.k * 2)
                return set_err(err, at + "conv weight bytes != c_out*c_in*k*k*2"), SN_E_INVALID;
            if (d.b_bytes != 0 && d.b_bytes != (int64_t)d.c_out * 2)
                return set_err(err, at + "bias bytes != c_out*2"), SN_E_INVALID;
            L.b_unit_bytes = d.b_bytes ? 2 : 0;
            out = image_slot(ho, wo, d.c_out);
            break;
        }
        case SN_OP_MAXPOOL: {
            if (d.k <= 0 || d.stride <= 0 || d.pad < 0 || d.pad >= d.k)
                return set_err(err, at + "bad pool geometry"), SN_E_INVALID;
            if (src->h != d.h_in || src->w != d.w_in || src->c != d.c_in || d.c_out != d.c_in)
                return set_err(err, at + "pool shape mismatch"), SN_E_INVALID;
            L.out_h = (d.h_in + 2 * d.pad - d.k) / d.stride + 1;
            L.out_w = (d.w_in + 2 * d.pad - d.k) / d.stride + 1;
            if (L.out_h <= 0 || L.out_w <= 0) return set_err(err, at + "empty output"), SN_E_INVALID;
            L.cin_p = src->cp;
            out = image_slot(L.out_h, L.out_w, d.c_in);
            break;
        }
        case SN_OP_GAVGPOOL:
            if (src->h != d.h_in || src->w != d.w_in || src->c != d.c_in || d.c_out != d.c_in)
                return set_err(err, at + "pool shape mismatch"), SN_E_INVALID;
            L.cin_p = src->cp;
            out = image_slot(1, 1, d.c_in);
            break;
        case SN_OP_UPSAMPLE_BILINEAR:
            if (d.scale <= 0 || src->h != d.h_in || src->w != d.w_in || src->c != d.c_in ||
                d.c_out != d.c_in)
                return set_err(err, at + "upsample shape mismatch"), SN_E_INVALID;
            L.cin_p = src->cp;
            L.out_h = d.h_in * d.scale;
            L.out_w = d.w_in * d.scale;
            out = image_slot(L.out_h, L.out_w, d.c_in);
            break;
        case SN_OP_LINEAR: {
            const bool swiglu = d.flags & SN_FLAG_SWIGLU;
            L.rows_per_unit = swiglu ? 2 : 1;
            if (swiglu && d.b_bytes) return set_err(err, at + "SwiGLU linear takes no bias"), SN_E_INVALID;
            if (!token) {
                if (d.flags & SN_FLAG_FLATTEN_CHW) {
                    if ((int64_t)src->c * src->h * src->w != d.c_in)
                        return set_err(err, at + "flatten: c_in != C*H*W of the input"), SN_E_INVALID;
                    if (src->h != d.h_in || src->w != d.w_in)
                        return set_err(err, at + "flatten: h_in/w_in mismatch"), SN_E_INVALID;
                    L.K = src->h * src->w * src->cp;
                } else {
                    if (src->rows != 1 || src->c != d.c_in)
                        return set_err(err, at + "linear input must be a vector of c_in"), SN_E_INVALID;
                    L.K = src->cp;
                }
                L.cin_p = src->cp;
                out = image_slot(1, 1, d.c_out);
                if (d.flags & SN_FLAG_OUT_F32) out.elem = 4;
            } else {
                if (src->c != d.c_in || d.c_in % 8)
                    return set_err(err, at + "token linear: c_in mismatch or not a multiple of 8"),
                           SN_E_INVALID;
                L.K = d.c_in;
                L.cin_p = d.c_in;
                int rows = (d.flags & SN_FLAG_LAST_ROW) ? 1 : max_tokens;
                out = token_slot(rows, d.c_out, (d.flags & SN_FLAG_OUT_F32) ? 4 : 2);
            }
            L.units = d.c_out;
            L.w_unit_bytes = (int64_t)L.K * 2 * L.rows_per_unit;
            if (d.w_bytes != (int64_t)d.c_out * L.rows_per_unit * d.c_in * 2)
                return set_err(err, at + "linear weight bytes != rows*c_in*2"), SN_E_INVALID;
            if (d.b_bytes != 0 && d.b_bytes != (int64_t)d.c_out * 2)
                return set_err(err, at + "bias bytes != c_out*2"), SN_E_INVALID;
            L.b_unit_bytes = d.b_bytes ? 2 : 0;
            break;
        }
        case SN_OP_EMBED:
            if (d.max_tokens <= 0) return set_err(err, at + "embed needs max_tokens"), SN_E_INVALID;
            if (d.c_in % 8) return set_err(err, at + "embedding width must be a multiple of 8"), SN_E_INVALID;
            if (d.w_bytes != (int64_t)d.c_out * d.c_in * 2)
                return set_err(err, at + "table bytes != vocab*d*2"), SN_E_INVALID;
            out = token_slot(max_tokens, d.c_in, 2);
            break;
        case SN_OP_RMSNORM:
            if (src->c != d.c_in || d.c_out != d.c_in)
                return set_err(err, at + "rmsnorm shape mismatch"), SN_E_INVALID;
            if (d.w_bytes != (int64_t)d.c_in * 2) return set_err(err, at + "gain bytes != d*2"), SN_E_INVALID;
            L.units = 1;
            L.w_unit_bytes = d.w_bytes;
            out = token_slot(src->rows, d.c_in, 2);
            break;
        case SN_OP_ATTENTION: {
            if (d.heads <= 0 || d.head_dim <= 0 || d.head_dim % 2 || d.kv_layer < 0 || d.max_seq <= 0)
                return set_err(err, at + "bad attention geometry"), SN_E_INVALID;
            if (d.head_dim < 8 || d.head_dim > 512 || (d.head_dim & (d.head_dim - 1)))
                return set_err(err, at + "head_dim must be a power of two in [8, 512]"), SN_E_UNSUPPORTED;
            int dm = d.heads * d.head_dim;
            if (src->c != 3 * dm || d.c_in != 3 * dm || d.c_out != dm)
                return set_err(err, at + "attention expects [T][3d] -> [T][d]"), SN_E_INVALID;
            out = token_slot(src->rows, dm, 2);
            break;
        }
        default:
            return set_err(err, at + "unknown op " + std::to_string(d.op)), SN_E_INVALID;
        }
        if (d.op != SN_OP_CONV2D && d.op != SN_OP_LINEAR && d.op != SN_OP_RMSNORM &&
            d.op != SN_OP_EMBED && (d.w_bytes || d.b_bytes))
            return set_err(err, at + "op takes no weights"), SN_E_INVALID;
        if (d.res >= 0) {
            const Slot *r = nullptr;
            int rc = use_slot(slots, d.res, li, err, &r);
            if (rc) return rc;
            if (!same_shape(*r, out)) return set_err(err, at + "residual shape != output shape"), SN_E_INVALID;
        }
        L.cout_p = out.cp;
        int rc = define_slot(slots, d.dst, out, li, err);
        if (rc) return rc;
    }
    return SN_OK;
}

// ---------------------------------------------------------------------------
// Prepack: canonical tensors -> device layout (once, at registration)
// ---------------------------------------------------------------------------
int prepack_layer(Layer &L, const uint8_t *blob, size_t blob_bytes, std::string &err) {
    const sn_layer &d = L.d;
    if ((uint64_t)d.w_off + (uint64_t)d.w_bytes > blob_bytes ||
        (uint64_t)d.b_off + (uint64_t)d.b_bytes > blob_bytes)
        return set_err(err, "weight offsets exceed the block buffer"), SN_E_INVALID;
    const uint16_t *w = (const uint16_t *)(blob + d.w_off);
    if ((d.w_off | d.b_off) & 1) return set_err(err, "weight offsets must be 2-byte aligned"), SN_E_INVALID;
    switch (d.op) {
    case SN_OP_CONV2D: {
        // [co][ci][r][s] -> [co][r][s][ci_p], zero padding channels
        const int co = d.c_out, ci = d.c_in, k = d.k, cp = L.cin_p;
        L.w_dev.assign((size_t)co * L.K, 0);
        for (int o = 0; o < co; ++o)
            for (int c = 0; c < ci; ++c)
                for (int r = 0; r < k; ++r)
                    for (int s = 0; s < k; ++s)
                        L.w_dev[(size_t)o * L.K + (r * k + s) * cp + c] =
                            w[(((size_t)o * ci + c) * k + r) * k + s];
        break;
    }
    case SN_OP_LINEAR: {
        const int n = d.c_out * L.rows_per_unit;
        L.w_dev.assign((size_t)n * L.K, 0);
        const bool swiglu = d.flags & SN_FLAG_SWIGLU;
        for (int row = 0; row < n; ++row) {
            // SwiGLU: device row 2j = W1 row j (gate), 2j+1 = W3 row j (up)
            int src_row = swiglu ? ((row & 1) ? d.c_out + row / 2 : row / 2) : row;
            const uint16_t *wr = w + (size_t)src_row * d.c_in;
            uint16_t *dr = L.w_dev.data() + (size_t)row * L.K;
            if (!L.token && (d.flags & SN_FLAG_FLATTEN_CHW)) {
                // canonical column c*H*W + h*W + x  ->  device column (h*W + x)*Cp + c
                const int H = d.h_in, W = d.w_in, C = d.c_in / (H * W), cp = L.cin_p;
                for (int c = 0; c < C; ++c)
                    for (int p = 0; p < H * W; ++p) dr[(size_t)p * cp + c] = wr[(size_t)c * H * W + p];
            } else {
                memcpy(dr, wr, (size_t)d.c_in * 2);
            }
        }
        break;
    }
    case SN_OP_RMSNORM:
    case SN_OP_EMBED:
        L.w_dev.assign(w, w + d.w_bytes / 2);
        break;
    default:
        break;
    }
    if (d.b_bytes) {
        const uint16_t *b = (const uint16_t *)(blob + d.b_off);
        L.b_dev.assign(b, b + d.b_bytes / 2);
    }
    return SN_OK;
}

// ---------------------------------------------------------------------------
// Slab lowering
// ---------------------------------------------------------------------------
namespace {
using PS = PieceSpec;

int64_t piece_bytes(const std::vector<Layer> &layers, const PS &p) {
    const Layer &L = layers[p.layer];
    if (!L.units || L.d.op == SN_OP_EMBED) return 0;
    int64_t n = p.u1 - p.u0;
    return align_up(n * L.w_unit_bytes) + align_up(n * L.b_unit_bytes);
}

int64_t slab_bytes(const std::vector<Layer> &layers, const SlabSpec &s) {
    int64_t b = 0;
    for (const PS &p : s) b += piece_bytes(layers, p);
    return b;
}

// Split slab s into two or more slabs; returns false if it cannot be split.
bool split_slab(const std::vector<Layer> &layers, const SlabSpec &s, int64_t target,
                std::vector<SlabSpec> &out) {
    std::vector<int> weighted;
    int64_t total = 0, biggest = 0;
    int wi = -1;
    for (int i = 0; i < (int)s.size(); ++i) {
        int64_t b = piece_bytes(layers, s[i]);
        if (b > 0) weighted.push_back(i);
        total += b;
        if (b > biggest && s[i].u1 - s[i].u0 >= 2) {
            biggest = b;
            wi = i;
        }
    }
    // A dominant layer (more than half the slab) is split by output channels,
    // with the rest of the slab attached to its first / last part; otherwise
    // the slab is cut at the layer boundary that balances the halves.
    const bool dominant = wi >= 0 && 2 * biggest > total;
    if (weighted.size() >= 2 && !dominant) {
        int64_t left = 0, best = -1;
        int cut = -1;
        for (int i = 0; i + 1 < (int)s.size(); ++i) {
            left += piece_bytes(layers, s[i]);
            if (i < weighted.front() || i >= weighted.back()) continue;
            int64_t worst = std::max(left, total - left);
            if (best < 0 || worst < best) {
                best = worst;
                cut = i + 1;
            }
        }
        if (cut < 0) return false;
        out.push_back(SlabSpec(s.begin(), s.begin() + cut));
        out.push_back(SlabSpec(s.begin() + cut, s.end()));
        return true;
    }
    if (wi < 0) return false;
    // split the chosen layer's output units into equal parts of <= target
    const PS &p = s[wi];
    const int64_t units = p.u1 - p.u0;
    if (units < 2) return false;
    const int64_t bytes = piece_bytes(layers, p);
    int64_t parts = std::max<int64_t>(2, (bytes + target - 1) / std::max<int64_t>(target, 1));
    parts = std::min(parts, units);
    for (int64_t k = 0; k < parts; ++k) {
        SlabSpec part;
        if (k == 0) part.insert(part.end(), s.begin(), s.begin() + wi);
        int64_t a = p.u0 + units * k / parts, b = p.u0 + units * (k + 1) / parts;
        part.push_back(PS{p.layer, a, b});
        if (k == parts - 1) part.insert(part.end(), s.begin() + wi + 1, s.end());
        out.push_back(part);
    }
    return true;
}
}  // namespace

// Balanced partition (Sec. 6: m = 2 blocks in flight, n = ceil(m s / b),
// rounded up to even): the layers of all blocks, in order, are cut into
// slabs of at most ceil(s / n) bytes (never more than half the budget, so any two consecutive
// slabs fit side by side); a layer that straddles a boundary is cut by
// output units, the part that fits closing the current slab.
static int balanced_slabs(const std::vector<Layer> &layers, int64_t B, int64_t max_slab,
                          std::vector<SlabSpec> &slabs, std::string &err) {
    int64_t total = 0;
    for (int li = 0; li < (int)layers.size(); ++li)
        total += piece_bytes(layers, PS{li, 0, layers[li].units ? layers[li].units : 0});
    int64_t cap = B / 2 / kAlign * kAlign;
    if (max_slab > 0) cap = std::min(cap, max_slab);
    if (cap <= 0) {
        err = "infeasible: budget too small to partition";
        return SN_E_INFEASIBLE;
    }
    // n even: slabs alternate between the two ends of the arena, so with an
    // even count the last slab sits at the other end from slab 0 and the next
    // inference's first swap-in overlaps the last slab's compute
    int64_t n = std::max<int64_t>(1, (2 * total + B - 1) / std::max<int64_t>(B, 1));
    if (n > 1 && (n & 1)) ++n;
    const int64_t target = std::min(cap, (total + n - 1) / n);
    slabs.clear();
    SlabSpec cur;
    int64_t acc = 0;
    auto close = [&]() {
        if (!cur.empty()) slabs.push_back(cur);
        cur.clear();
        acc = 0;
    };
    for (int li = 0; li < (int)layers.size(); ++li) {
        const Layer &L = layers[li];
        int64_t u0 = 0;
        const int64_t u1 = L.units ? L.units : 0;
        for (;;) {
            const int64_t b = piece_bytes(layers, PS{li, u0, u1});
            if (acc + b <= target || b == 0) {
                cur.push_back(PS{li, u0, u1});
                acc += b;
                break;
            }
            // the largest number of units that still fits the current slab
            int64_t lo = 0, hi = u1 - u0;
            const bool splittable = L.units && L.d.op != SN_OP_EMBED && hi >= 2;
            if (splittable) {
                while (lo < hi) {
                    const int64_t mid = (lo + hi + 1) / 2;
                    if (acc + piece_bytes(layers, PS{li, u0, u0 + mid}) <= target) lo = mid;
                    else hi = mid - 1;
                }
            }
            if (lo > 0) {
                cur.push_back(PS{li, u0, u0 + lo});
                u0 += lo;
                close();
                continue;
            }
            if (!cur.empty()) {
                close();
                continue;
            }
            // an empty slab cannot take it: one unit is larger than the target
            if (b > cap && !splittable) {
                err = "infeasible: layer " + std::to_string(li) + " (" + std::to_string(b) +
                      " bytes) exceeds half the budget and cannot be split";
                return SN_E_INFEASIBLE;
            }
            const int64_t one = piece_bytes(layers, PS{li, u0, u0 + 1});
            if (one > cap) {
                err = "infeasible: one output unit of layer " + std::to_string(li) +
                      " exceeds half the budget";
                return SN_E_INFEASIBLE;
            }
            // fill up to the cap instead of the target
            int64_t k = 1;
            while (u0 + k < u1 && piece_bytes(layers, PS{li, u0, u0 + k + 1}) <= cap) ++k;
            cur.push_back(PS{li, u0, u0 + k});
            u0 += k;
            close();
            if (u0 >= u1) break;
        }
    }
    close();
    // alignment padding can leave a small remainder slab: fold it into the
    // previous one when that stays within half the budget
    if (slabs.size() >= 2) {
        const int64_t last = slab_bytes(layers, slabs.back());
        const int64_t prev = slab_bytes(layers, slabs[slabs.size() - 2]);
        if (4 * last < target && prev + last <= cap) {
            SlabSpec &p = slabs[slabs.size() - 2];
            p.insert(p.end(), slabs.back().begin(), slabs.back().end());
            slabs.pop_back();
        }
    }
    return SN_OK;
}

int64_t spec_bytes(const std::vector<Layer> &layers, const SlabSpec &s) { return slab_bytes(layers, s); }

// Lowering of partitions 0 and 1: start from the user blocks (0) or the
// balanced re-cut (1), then split until every slab and every two consecutive
// slabs fit.
static int lower_slabs(const std::vector<Layer> &layers, int n_blocks, int64_t B, int64_t max_slab,
                       bool balanced, std::vector<SlabSpec> &slabs, std::string &err) {
    slabs.assign(n_blocks, SlabSpec());
    for (int li = 0; li < (int)layers.size(); ++li) {
        const Layer &L = layers[li];
        int64_t u1 = L.units ? L.units : 0;
        slabs[L.block].push_back(PS{li, 0, u1});
    }
    if (balanced) {
        int64_t total = 0;
        for (const SlabSpec &ss : slabs) total += slab_bytes(layers, ss);
        // a model that fits stays as the user gave it (the run is resident)
        if (total > B) {
            int rc = balanced_slabs(layers, B, max_slab, slabs, err);
            if (rc) return rc;
        }
    }
    for (int iter = 0; iter < 1000000; ++iter) {
        const int n = (int)slabs.size();
        std::vector<int64_t> sz(n);
        for (int i = 0; i < n; ++i) sz[i] = slab_bytes(layers, slabs[i]);
        int j = -1;
        int64_t target = B / 2;
        for (int i = 0; i < n && j < 0; ++i) {
            if (sz[i] > B) {
                j = i;
            } else if (max_slab > 0 && sz[i] > max_slab) {
                j = i;
                target = max_slab;
            }
        }
        int other = -1;
        for (int i = 0; i + 1 < n && j < 0; ++i) {
            if (sz[i] + sz[i + 1] > B) {
                j = sz[i] >= sz[i + 1] ? i : i + 1;
                other = sz[i] >= sz[i + 1] ? i + 1 : i;
            }
        }
        if (j < 0) break;
        std::vector<SlabSpec> parts;
        if (!split_slab(layers, slabs[j], target, parts)) {
            if (other >= 0 && split_slab(layers, slabs[other], target, parts)) {
                j = other;
            } else {
                err = "infeasible: slab of " + std::to_string(sz[j]) +
                      " bytes cannot be split further to meet the budget (" + std::to_string(B) +
                      " bytes for two consecutive slabs)";
                return SN_E_INFEASIBLE;
            }
        }
        slabs.erase(slabs.begin() + j);
        slabs.insert(slabs.begin() + j, parts.begin(), parts.end());
    }
    return SN_OK;
}

int plan_slabs(const std::vector<Layer> &layers, int n_blocks, int64_t split_budget,
               int64_t arena_budget, int64_t max_slab, int partition, const CostModel &cost,
               PlanResult &res, std::string &err) {
    const int64_t B = split_budget / kAlign * kAlign;
    std::vector<SlabSpec> slabs;
    int rc = lower_slabs(layers, n_blocks, B, max_slab, partition == 1, slabs, err);
    if (rc) return rc;
    if (partition == 2) {
        int64_t total = 0;
        for (const SlabSpec &ss : slabs) total += slab_bytes(layers, ss);
        if (total > B) {
            // the user blocks and the balanced partition compete with the
            // searched ones
            std::vector<std::vector<SlabSpec>> seeds{slabs};
            std::vector<SlabSpec> bal;
            std::string ignored;
            if (!lower_slabs(layers, n_blocks, B, max_slab, true, bal, ignored)) seeds.push_back(bal);
            std::vector<SlabSpec> found;
            rc = search_partition(layers, B, arena_budget, max_slab, cost, seeds, found, err);
            if (rc) return rc;
            slabs.swap(found);
        }
    }
    layout_slabs(layers, slabs, res);
    return SN_OK;
}

// Lay out each slab: every tensor 256-byte aligned, slabs back to back in the
// image.
void layout_slabs(const std::vector<Layer> &layers, const std::vector<SlabSpec> &slabs,
                  PlanResult &res) {
    res.pieces.clear();
    res.slabs.clear();
    int64_t image_off = 0;
    for (const SlabSpec &ss : slabs) {
        Slab sl;
        int64_t off = 0;
        for (const PS &p : ss) {
            Piece pc;
            pc.layer = p.layer;
            pc.u0 = p.u0;
            pc.u1 = p.u1;
            const Layer &L = layers[p.layer];
            if (L.units && L.d.op != SN_OP_EMBED) {
                int64_t n = p.u1 - p.u0;
                pc.w_bytes = n * L.w_unit_bytes;
                pc.w_off = off;
                off += align_up(pc.w_bytes);
                if (L.b_unit_bytes) {
                    pc.b_bytes = n * L.b_unit_bytes;
                    pc.b_off = off;
                    off += align_up(pc.b_bytes);
                }
            }
            sl.pieces.push_back((int)res.pieces.size());
            res.pieces.push_back(pc);
        }
        sl.bytes = off;
        sl.image_off = image_off;
        image_off += off;
        res.slabs.push_back(sl);
    }
    res.image_bytes = image_off;
}

// Arena placement.  The pair constraint (Eq. 3) guarantees that slab i and
// slab i+1 fit side by side at the two ends of the arena; within that
// guarantee each slab is put where its swap-in has to wait for the oldest
// possible earlier slab, so that small slabs let the DMA run several slabs
// ahead of the compute (the m = 2 parallel blocks of Sec. 6.2.2 are the
// floor, not the ceiling).  A position in the middle of the arena is taken
// only if the next slab still fits at one of the two ends beside it, which
// keeps every later placement feasible.
int place_slabs(PlanResult &p, int64_t arena_budget, std::string &err) {
    const int64_t B = arena_budget / kAlign * kAlign;
    const int n = (int)p.slabs.size();
    if (p.image_bytes <= B) {
        p.resident = true;
        int64_t off = 0;
        for (Slab &s : p.slabs) {
            s.arena_off = off;
            s.wait = -1;
            off += s.bytes;
        }
        p.high_water = off;
        return SN_OK;
    }
    p.resident = false;
    p.high_water = 0;
    auto overlap = [](int64_t a, int64_t sa, int64_t b, int64_t sb) {
        return sa > 0 && sb > 0 && a < b + sb && b < a + sa;
    };
    for (int i = 0; i < n; ++i) {
        Slab &s = p.slabs[i];
        if (s.bytes > B || (i + 1 < n && s.bytes + p.slabs[i + 1].bytes > B)) {
            err = "infeasible: slabs " + std::to_string(i) + "," + std::to_string(i + 1) +
                  " do not fit the arena together";
            return SN_E_INFEASIBLE;
        }
        std::vector<int64_t> cand = {0, B - s.bytes};
        for (int j = 0; j < i; ++j) {
            cand.push_back(p.slabs[j].arena_off + p.slabs[j].bytes);
            cand.push_back(p.slabs[j].arena_off - s.bytes);
        }
        const int64_t next = i + 1 < n ? p.slabs[i + 1].bytes : 0;
        int best_wait = 1 << 30;
        int64_t best_off = -1;
        bool best_clear0 = false;
        for (int64_t c : cand) {
            if (c < 0 || c + s.bytes > B || c % kAlign) continue;
            if (i > 0 && overlap(c, s.bytes, p.slabs[i - 1].arena_off, p.slabs[i - 1].bytes)) continue;
            const bool at_end = c == 0 || c == B - s.bytes;
            if (!at_end && next > 0 && !(next <= c || c + s.bytes + next <= B)) continue;
            int w = -1;
            for (int j = i - 1; j >= 0; --j)
                if (overlap(c, s.bytes, p.slabs[j].arena_off, p.slabs[j].bytes)) {
                    w = j;
                    break;
                }
            // ties: keep clear of slab 0's range (the next inference's first
            // swap-in then need not wait for this slab), then the lowest offset
            const bool clear0 = i == 0 || !overlap(c, s.bytes, p.slabs[0].arena_off, p.slabs[0].bytes);
            if (w < best_wait || (w == best_wait && clear0 && !best_clear0) ||
                (w == best_wait && clear0 == best_clear0 && c < best_off)) {
                best_wait = w;
                best_off = c;
                best_clear0 = clear0;
            }
        }
        if (best_off < 0) {
            err = "placement failed for slab " + std::to_string(i);
            return SN_E_INFEASIBLE;
        }
        s.arena_off = best_off;
        s.wait = best_wait;
        p.high_water = std::max(p.high_water, s.arena_off + s.bytes);
    }
    // Back-to-back inferences: a slab whose range no earlier slab of the same
    // inference uses is overwritten, one inference later, only after the last
    // slab that shares its range has run, so its swap-in can start while the
    // previous inference is still computing its remaining slabs.
    for (int j = 0; j < n; ++j) {
        Slab &s = p.slabs[j];
        s.wrap = -1;
        if (s.wait >= 0) continue;
        for (int i = n - 1; i > j; --i)
            if (overlap(s.arena_off, s.bytes, p.slabs[i].arena_off, p.slabs[i].bytes)) {
                s.wrap = i;
                break;
            }
    }
    return SN_OK;
}

// Activation slots share one pool: a slot's bytes are reused once its last
// reader has run.  A slot is live over [first writer, last reader]; two slots
// may share memory only if their live ranges do not touch (a layer never
// writes over a buffer it reads).
void assign_slot_offsets(std::vector<Slot> &slots, int64_t &total) {
    std::vector<int> order;
    for (int i = 0; i < (int)slots.size(); ++i)
        if (slots[i].used) {
            slots[i].bytes = align_up((int64_t)slots[i].rows * slots[i].cp * slots[i].elem);
            order.push_back(i);
        }
    std::sort(order.begin(), order.end(), [&](int a, int b) {
        return slots[a].first != slots[b].first ? slots[a].first < slots[b].first : a < b;
    });
    std::vector<int> placed;
    total = 0;
    for (int id : order) {
        Slot &s = slots[id];
        std::vector<std::pair<int64_t, int64_t>> busy;
        for (int q : placed) {
            const Slot &o = slots[q];
            if (!(o.last < s.first || s.last < o.first)) busy.push_back({o.off, o.off + o.bytes});
        }
        std::sort(busy.begin(), busy.end());
        int64_t off = 0;
        for (auto &b : busy) {
            if (off + s.bytes <= b.first) break;
            off = std::max(off, b.second);
        }
        s.off = off;
        total = std::max(total, off + s.bytes);
        placed.push_back(id);
    }
}

void write_image(const std::vector<Layer> &layers, const PlanResult &p, uint8_t *image) {
    memset(image, 0, (size_t)p.image_bytes);
    for (const Slab &s : p.slabs) {
        for (int pi : s.pieces) {
            const Piece &pc = p.pieces[pi];
            const Layer &L = layers[pc.layer];
            if (pc.w_bytes) {
                const uint8_t *src = (const uint8_t *)L.w_dev.data() + pc.u0 * L.w_unit_bytes;
                memcpy(image + s.image_off + pc.w_off, src, (size_t)pc.w_bytes);
            }
            if (pc.b_bytes) {
                const uint8_t *src = (const uint8_t *)L.b_dev.data() + pc.u0 * L.b_unit_bytes;
                memcpy(image + s.image_off + pc.b_off, src, (size_t)pc.b_bytes);
            }
        }
    }
}

}  // namespace sn
