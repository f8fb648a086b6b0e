// Pre-processor of the initialization stage (Sec. 3.2.1, Eq. 6-8) and the
// default auxiliary network (Sec. 3.2.2).  Host code only: it runs once,
// before training, on the server.
//
// A network is a table of units the split may follow (a convolution with
// its normalisation and activation, a pooling layer, a fully connected
// layer, a MobileNetV3 bottleneck, an embedding, a transformer encoder
// layer; blocks are never cut).  Per unit and sample: forward FLOPs of its
// convolutions and matrix products (2 per multiply-add; normalisation,
// activations, pooling and softmax not counted), parameters, output values.
// Eq. 6-8 then take O_l = 3 x forward FLOPs x batch (forward, input- and
// weight-gradient products of an iteration) and S_l = output values x batch
// x bytes per value.
#include <algorithm>
#include <cmath>

#include "common.h"

namespace {

fo_unit unit(int32_t kind) {
    fo_unit u{};
    u.kind = kind;
    u.stride = 1;
    return u;
}

int32_t out_side(int32_t in, int32_t k, int32_t stride) { return (in + 2 * (k / 2) - k) / stride + 1; }

fo_unit conv_unit(int32_t k, int32_t stride, int32_t ci, int32_t co, int32_t h, int32_t w, bool bias, bool norm) {
    fo_unit u = unit(FO_UNIT_CONV);
    u.k = k;
    u.stride = stride;
    u.c_in = ci;
    u.c_out = co;
    u.h_out = out_side(h, k, stride);
    u.w_out = out_side(w, k, stride);
    u.norm = norm;
    u.params = (int64_t)k * k * ci * co + (bias ? co : 0) + (norm ? 2 * co : 0);
    u.fwd_flops = 2.0 * k * k * ci * co * u.h_out * u.w_out;
    u.out_elems = (double)co * u.h_out * u.w_out;
    return u;
}

// size 0: global average pool
fo_unit pool_unit(int32_t c, int32_t h, int32_t w, int32_t size) {
    fo_unit u = unit(FO_UNIT_POOL);
    u.c_in = u.c_out = c;
    u.k = u.stride = size == 0 ? 1 : size;
    if (size == 0) u.k = 0;
    u.h_out = size == 0 ? 1 : h / size;
    u.w_out = size == 0 ? 1 : w / size;
    u.out_elems = (double)c * u.h_out * u.w_out;
    return u;
}

fo_unit fc_unit(int32_t ci, int32_t co) {
    fo_unit u = unit(FO_UNIT_FC);
    u.c_in = ci;
    u.c_out = co;
    u.h_out = u.w_out = 1;
    u.params = (int64_t)ci * co + co;
    u.fwd_flops = 2.0 * ci * co;
    u.out_elems = co;
    return u;
}

// squeeze width of a MobileNetV3 squeeze-excitation: expansion / 4 rounded to a
// multiple of 8, at least 8 and not below 90% of the unrounded width
int32_t squeeze_width(int32_t expand) {
    const int32_t v = expand / 4;
    int32_t n = std::max(8, (v + 4) / 8 * 8);
    if (n < 0.9 * v) n += 8;
    return n;
}

// expansion 1x1 (absent when expand == ci), depthwise k x k, optional
// squeeze-excitation (two 1x1 layers with bias on the pooled vector),
// projection 1x1; a batch norm after each convolution
fo_unit bneck_unit(int32_t k, int32_t e, int32_t ci, int32_t co, bool se, int32_t stride, int32_t h, int32_t w) {
    fo_unit u = unit(FO_UNIT_BNECK);
    u.k = k;
    u.stride = stride;
    u.c_in = ci;
    u.c_out = co;
    u.expand = e;
    u.norm = 1;
    u.se = se;
    u.h_out = out_side(h, k, stride);
    u.w_out = out_side(w, k, stride);
    const double hw_in = (double)h * w, hw_out = (double)u.h_out * u.w_out;
    int64_t p = 0;
    double f = 0;
    if (e != ci) {
        p += (int64_t)ci * e + 2 * e;
        f += 2.0 * ci * e * hw_in;
    }
    p += (int64_t)k * k * e + 2 * e;
    f += 2.0 * k * k * e * hw_out;
    if (se) {
        const int32_t s = squeeze_width(e);
        p += (int64_t)e * s + s + (int64_t)s * e + e;
        f += 2.0 * ((double)e * s + (double)s * e);
    }
    p += (int64_t)e * co + 2 * co;
    f += 2.0 * e * co * hw_out;
    u.params = p;
    u.fwd_flops = f;
    u.out_elems = (double)co * hw_out;
    return u;
}

fo_unit emb_unit(int32_t d, int32_t seq) {
    fo_unit u = unit(FO_UNIT_EMB);
    u.c_out = d;
    u.h_out = seq;
    u.w_out = 1;
    u.out_elems = (double)d * seq;
    return u;
}

// post-norm encoder layer: fused q, k, v projection, attention over seq
// positions, output projection, two-layer FFN, two LayerNorms
fo_unit enc_unit(int32_t d, int32_t heads, int32_t hidden, int32_t seq) {
    fo_unit u = unit(FO_UNIT_ENC);
    u.c_in = u.c_out = d;
    u.heads = heads;
    u.hidden = hidden;
    u.norm = 1;
    u.h_out = seq;
    u.w_out = 1;
    u.params = 4LL * d * d + 4 * d + 2 * d + (int64_t)d * hidden + hidden + (int64_t)hidden * d + d + 2 * d;
    const double L = seq;
    u.fwd_flops = 2.0 * L * d * 3 * d + 2.0 * L * L * d * 2 + 2.0 * L * d * d + 2.0 * L * d * hidden * 2;
    u.out_elems = (double)d * seq;
    return u;
}

struct Bneck {
    int32_t k, e, co;
    bool se;
    int32_t s;
};
// MobileNetV3-Large's bottlenecks (Table 4 with the expansions, strides and
// squeeze-excitation placement of the architecture's own definition)
const Bneck kMbv3Large[] = {
    {3, 16, 16, false, 1},  {3, 64, 24, false, 2},  {3, 72, 24, false, 1},  {5, 72, 40, true, 2},
    {5, 120, 40, true, 1},  {5, 120, 40, true, 1},  {3, 240, 80, false, 2}, {3, 200, 80, false, 1},
    {3, 184, 80, false, 1}, {3, 184, 80, false, 1}, {3, 480, 112, true, 1}, {3, 672, 112, true, 1},
    {5, 672, 160, true, 2}, {5, 960, 160, true, 1}, {5, 960, 160, true, 1},
};

struct Table {
    fo_unit* out;
    int32_t max, n = 0;
    void add(const fo_unit& u) {
        if (n < max) out[n] = u;
        n++;
    }
    const fo_unit& last() const { return last_u; }
    fo_unit last_u{};
    void push(const fo_unit& u) {
        add(u);
        last_u = u;
    }
};

}  // namespace

extern "C" int32_t fo_net_units(int32_t net, int32_t classes, int32_t in_hw, fo_unit* out, int32_t max_units) {
    if (classes < 1 || in_hw < 1 || max_units < 0 || (max_units > 0 && !out)) {
        fo::set_error("fo_net_units: classes=%d, in_hw=%d, max_units=%d", classes, in_hw, max_units);
        return -1;
    }
    Table t{out, max_units};
    switch (net) {
        case FO_NET_VGG5: {
            if (in_hw % 8) break;
            int32_t h = in_hw;
            const int32_t ch[4] = {3, 32, 64, 64};
            for (int i = 0; i < 3; ++i) {
                t.push(conv_unit(3, 1, ch[i], ch[i + 1], h, h, false, true));
                t.push(pool_unit(ch[i + 1], h, h, 2));
                h /= 2;
            }
            t.push(fc_unit(64 * h * h, 128));
            t.push(fc_unit(128, classes));
            return t.n;
        }
        case FO_NET_VGG16: {
            if (in_hw % 32) break;
            const int32_t plan[] = {64, 64, 0, 128, 128, 0, 256, 256, 256, 0, 512, 512, 512, 0, 512, 512, 512, 0};
            int32_t h = in_hw, c = 3;
            for (int32_t v : plan) {
                if (v == 0) {
                    t.push(pool_unit(c, h, h, 2));
                    h /= 2;
                } else {
                    t.push(conv_unit(3, 1, c, v, h, h, true, false));
                    c = v;
                }
            }
            t.push(fc_unit(c * h * h, 512));
            t.push(fc_unit(512, 512));
            t.push(fc_unit(512, classes));
            return t.n;
        }
        case FO_NET_MOBILENETV3_LARGE: {
            t.push(conv_unit(3, 2, 3, 16, in_hw, in_hw, false, true));
            int32_t h = t.last().h_out, c = 16;
            for (const Bneck& b : kMbv3Large) {
                t.push(bneck_unit(b.k, b.e, c, b.co, b.se, b.s, h, h));
                h = t.last().h_out;
                c = b.co;
            }
            t.push(conv_unit(1, 1, c, 960, h, h, false, true));
            t.push(pool_unit(960, h, h, 0));
            t.push(fc_unit(960, 1280));
            t.push(fc_unit(1280, classes));
            return t.n;
        }
        case FO_NET_TRANSFORMER6:
        case FO_NET_TRANSFORMER12: {
            const bool six = net == FO_NET_TRANSFORMER6;
            t.push(emb_unit(100, in_hw));
            for (int i = 0; i < (six ? 6 : 12); ++i) t.push(enc_unit(100, six ? 5 : 50, 100, in_hw));
            t.push(fc_unit(100, classes));
            return t.n;
        }
        default:
            fo::set_error("fo_net_units: unknown network %d", net);
            return -1;
    }
    fo::set_error("fo_net_units: network %d needs in_hw divisible by its total pooling (got %d)", net, in_hw);
    return -1;
}

extern "C" fo_status fo_select_split(const fo_unit* units, int32_t L, int32_t batch, int32_t bytes_per_value,
                                     int32_t K, const double* flops_per_s, const double* bytes_per_s,
                                     double* cost_out, int32_t* split_out) {
    FO_CHECK(units && L >= 1 && split_out, "fo_select_split: no units");
    FO_CHECK(batch >= 1 && bytes_per_value >= 1, "fo_select_split: batch=%d, bytes_per_value=%d", batch,
             bytes_per_value);
    FO_CHECK(K >= 1 && flops_per_s && bytes_per_s, "fo_select_split: no devices");
    for (int32_t k = 0; k < K; ++k)
        FO_CHECK(flops_per_s[k] > 0 && bytes_per_s[k] > 0, "fo_select_split: device %d: o=%g, b=%g", k,
                 flops_per_s[k], bytes_per_s[k]);
    double prefix = 0.0, best = 0.0;
    int32_t arg = 0;
    for (int32_t l = 0; l < L; ++l) {
        prefix += 3.0 * units[l].fwd_flops * batch;                       // sum_{i<=l} O_i (Eq. 6)
        const double S = units[l].out_elems * batch * bytes_per_value;    // S_l
        double worst = 0.0;
        for (int32_t k = 0; k < K; ++k) {                                  // max over devices of Eq. 6, 7
            const double c = std::max(prefix / flops_per_s[k], S / bytes_per_s[k]);
            if (k == 0 || c > worst) worst = c;
        }
        if (cost_out) cost_out[l] = worst;
        if (l == 0 || worst < best) {                                      // Eq. 8, first minimum
            best = worst;
            arg = l;
        }
    }
    *split_out = arg + 1;
    return FO_OK;
}

extern "C" int32_t fo_aux_network(const fo_unit* units, int32_t L, int32_t split, int32_t classes, fo_unit* out,
                                  int32_t max_units) {
    if (!units || split < 1 || split > L || classes < 1 || max_units < 0 || (max_units > 0 && !out)) {
        fo::set_error("fo_aux_network: split=%d of %d units, classes=%d", split, L, classes);
        return -1;
    }
    int32_t j = split - 1;
    while (j >= 0 && units[j].kind == FO_UNIT_POOL) --j;  // the last unit of M_d with parameters
    if (j < 0) {
        fo::set_error("fo_aux_network: no unit with parameters before the split");
        return -1;
    }
    const fo_unit& last = units[j];
    const fo_unit& o = units[split - 1];
    Table t{out, max_units};
    switch (last.kind) {
        case FO_UNIT_CONV:
            t.push(conv_unit(last.k, 1, o.c_out, o.c_out, o.h_out, o.w_out, true, last.norm != 0));
            t.push(pool_unit(o.c_out, o.h_out, o.w_out, 0));
            t.push(fc_unit(o.c_out, classes));
            return t.n;
        case FO_UNIT_BNECK:
            t.push(bneck_unit(last.k, last.expand, o.c_out, o.c_out, last.se != 0, 1, o.h_out, o.w_out));
            t.push(pool_unit(o.c_out, o.h_out, o.w_out, 0));
            t.push(fc_unit(o.c_out, classes));
            return t.n;
        case FO_UNIT_ENC:
            t.push(enc_unit(last.c_out, last.heads, last.hidden, last.h_out));
            t.push(fc_unit(last.c_out, classes));
            return t.n;
        case FO_UNIT_EMB:
            t.push(fc_unit(last.c_out, classes));
            return t.n;
        case FO_UNIT_FC:
            t.push(fc_unit(last.c_out, last.c_out));
            t.push(fc_unit(last.c_out, classes));
            return t.n;
        default:
            fo::set_error("fo_aux_network: unit kind %d", last.kind);
            return -1;
    }
}
