// Model description, service profile (Eq. 1-4), workspace layout and the
// sliced executor: slices run op by op on one stream, RD ops as k
// sub-slices of one launch, and slice boundaries pass through the codec.
#include <algorithm>
#include <cmath>
#include <map>
#include <string>
#include <vector>

#include "internal.h"

namespace mopar {

int plan_slices_impl(const mopar_layer_profile* L, int32_t n, const mopar_plan_opts* o, mopar_plan* out);

namespace {

constexpr double kPeakBf16 = 2.5e15, kPeakF32 = 157.3e12, kPeakBytes = 8.0e12;

int64_t numel(const mopar_tensor_desc& t) {
    int64_t n = 1;
    for (int i = 0; i < t.rank; ++i) n *= t.dims[i];
    return n;
}

size_t elt_bytes(int dtype) { return dtype == MOPAR_BF16 ? 2 : 4; }

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

struct TempReq {
    size_t bytes;
};

}  // namespace

struct OpInfo {
    int splits = 1;                // conv / linear: split-K factor of the GEMM
    int partial_temp = -1;         // index into temps of the split-K partial sums
    int ctr_temp = -1;             // index into temps of the 256 x 256 GEMM tile counters
    int cs = 0;                    // conv: input channel storage stride (padded for the model input)
    bool input_is_model = false;   // conv: reads the NCHW float32 model input
    int64_t K = 0, M = 0;          // GEMM sizes (conv / linear)
    std::vector<size_t> temps;     // scratch buffers needed while this op runs
    std::vector<size_t> temp_off;  // their workspace offsets
};

}  // namespace mopar

struct mopar_model_s {
    int dtype;
    std::vector<mopar_tensor_desc> tensors;
    std::vector<mopar_op> ops;
    std::vector<mopar::OpInfo> info;
    int n_layers;
    int input, output;
    const unsigned char* weights;
    size_t weights_bytes;
    std::vector<int> layer_first, layer_last;   // op index range per planning node
    std::vector<int> layer_out;                 // tensor leaving each node
    std::vector<std::vector<int>> cross;        // per cut j (after node j): node outputs of nodes <= j
                                                // that nodes > j read, ascending tensor id
    std::vector<size_t> offset;                 // workspace offset per tensor (SIZE_MAX: not in ws)
    size_t ws_bytes;
    // measurement (timing slots: ops, then encode / decode per cut): each kernel launched
    // inside a slot gets an event pair from kev; a slot owns the pairs [slot_lo, slot_hi)
    bool timing = false;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> kev;
    size_t kev_next = 0;
    std::vector<size_t> slot_lo, slot_hi;
    void free_events() {
        for (auto& e : kev) {
            (void)hipEventDestroy(e.first);
            (void)hipEventDestroy(e.second);
        }
        kev.clear();
        kev_next = 0;
    }
    ~mopar_model_s() { free_events(); }
};

namespace mopar {

thread_local LaunchTimer* t_timer = nullptr;

namespace {


bool shape_eq(const mopar_tensor_desc& t, std::initializer_list<int64_t> d) {
    if (t.rank != static_cast<int>(d.size())) return false;
    int i = 0;
    for (int64_t v : d)
        if (t.dims[i++] != v) return false;
    return true;
}

std::string op_name(const mopar_model_s& m, int i) {
    return "op " + std::to_string(i) + " (kind " + std::to_string(m.ops[i].kind) + ")";
}

// parameter element count of an op (logical shapes; conv counts C, not the padded Cs)
int64_t param_elems(const mopar_model_s& m, const mopar_op& op) {
    const auto& in = m.tensors[op.in0];
    switch (op.kind) {
        case MOPAR_OP_CONV: return static_cast<int64_t>(op.n_out) * in.dims[1] * op.kh * op.kw + op.n_out;
        case MOPAR_OP_LINEAR: {
            const int64_t K = in.rank == 4 ? in.dims[1] * in.dims[2] * in.dims[3] : in.dims[in.rank - 1];
            return static_cast<int64_t>(op.n_out) * K + op.n_out;
        }
        case MOPAR_OP_LAYERNORM: return 2 * in.dims[in.rank - 1];
        case MOPAR_OP_EMBED_BERT: {
            const int64_t f = m.tensors[op.out].dims[2];
            return (op.rows[0] + op.rows[1] + op.rows[2]) * f + 2 * f;
        }
        case MOPAR_OP_EMBED: return op.rows[0] * m.tensors[op.out].dims[2];
        case MOPAR_OP_LSTM: {
            const int64_t e = in.dims[2], h = op.n_out;
            return 4 * h * e + 4 * h * h + 8 * h;
        }
        default: return 0;
    }
}

}  // namespace

// Operator profile: memory = bytes of parameters + inputs + output; time =
// max(FLOP / peak, bytes / HBM bandwidth); FLOP only for contractions.
static void op_profile(const mopar_model_s& m, const mopar_op& op, double* mem, double* time) {
    const int64_t pb = param_elems(m, op) * static_cast<int64_t>(elt_bytes(m.dtype));
    int64_t ib = numel(m.tensors[op.in0]) * static_cast<int64_t>(elt_bytes(m.tensors[op.in0].dtype));
    if (op.in1 >= 0) ib += numel(m.tensors[op.in1]) * static_cast<int64_t>(elt_bytes(m.tensors[op.in1].dtype));
    const auto& o = m.tensors[op.out];
    // a conv that fills part of a concatenated tensor counts its own channels only
    const int64_t on = op.kind == MOPAR_OP_CONV ? numel(o) / o.dims[1] * op.n_out : numel(o);
    const int64_t ob = on * static_cast<int64_t>(elt_bytes(o.dtype));
    const auto& in = m.tensors[op.in0];
    int64_t flop = 0;
    switch (op.kind) {
        case MOPAR_OP_CONV: flop = 2 * on * in.dims[1] * op.kh * op.kw; break;
        case MOPAR_OP_LINEAR: {
            const int64_t K = in.rank == 4 ? in.dims[1] * in.dims[2] * in.dims[3] : in.dims[in.rank - 1];
            flop = 2 * numel(o) * K;
            break;
        }
        case MOPAR_OP_ATTENTION: flop = 4 * o.dims[0] * o.dims[1] * o.dims[1] * o.dims[2]; break;
        case MOPAR_OP_LSTM: flop = 2 * o.dims[0] * o.dims[1] * 4 * o.dims[2] * (in.dims[2] + o.dims[2]); break;
        default: break;
    }
    *mem = static_cast<double>(pb + ib + ob);
    const double peak = m.dtype == MOPAR_BF16 ? kPeakBf16 : kPeakF32;
    *time = std::fmax(static_cast<double>(flop) / peak, *mem / kPeakBytes);
}

int model_profile_impl(const mopar_model_s* m, mopar_layer_profile* out, double frac) {
    if (!m || !out) return set_error(MOPAR_E_ARG, "mopar_model_profile: null argument");
    if (!(frac > 0.0 && frac <= 1.0)) return set_error(MOPAR_E_ARG, "mopar_model_profile_dominant: frac must be in (0, 1]");
    for (int l = 0; l < m->n_layers; ++l) {
        double mc = 0.0, tc = 0.0;
        std::map<int, std::vector<std::pair<int, int>>> at_pos;   // pos -> (branch, op)
        int rdw = 0;
        // dominant operators: largest footprints first, the shortest prefix reaching frac
        const int f0 = m->layer_first[l], nl = m->layer_last[l] - f0 + 1;
        std::vector<double> mem(nl);
        double total = 0.0;
        for (int q = 0; q < nl; ++q) {
            double tt;
            op_profile(*m, m->ops[f0 + q], &mem[q], &tt);
            total = total + mem[q];
        }
        std::vector<int> order(nl);
        for (int q = 0; q < nl; ++q) order[q] = q;
        std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return mem[a] > mem[b]; });
        std::vector<char> keep(nl, frac >= 1.0 ? 1 : 0);
        if (frac < 1.0) {
            double acc = 0.0;
            for (int q : order) {
                acc = acc + mem[q];
                keep[q] = 1;
                if (acc >= frac * total) break;
            }
        }
        for (int i = m->layer_first[l]; i <= m->layer_last[l]; ++i) {
            const auto& op = m->ops[i];
            if (op.rd) rdw = rdw == 0 ? op.n_out : std::min(rdw, op.n_out);
            if (!keep[i - f0]) continue;
            if (op.branch == 0) {
                double mm, tt;
                op_profile(*m, op, &mm, &tt);
                mc = std::fmax(mc, mm);
                tc = tc + tt;
            } else {
                at_pos[op.pos].push_back({op.branch, i});
            }
        }
        double mb = 0.0, tb = 0.0;
        for (auto& kv : at_pos) {                    // positions ascending
            auto v = kv.second;
            std::stable_sort(v.begin(), v.end(), [](auto a, auto b) { return a.first < b.first; });
            double sm = 0.0, mt = 0.0;
            for (auto& bo : v) {
                double mm, tt;
                op_profile(*m, m->ops[bo.second], &mm, &tt);
                sm = sm + mm;
                mt = std::fmax(mt, tt);
            }
            mb = std::fmax(mb, sm);
            tb = tb + mt;
        }
        out[l].mem_bytes = std::fmax(mc, mb);
        out[l].time_s = tc + tb;
        // bytes a cut after this node moves: every tensor crossing it (the parallel edges of
        // Sec. III-C's edge elimination merged, sizes summed in tensor-id order)
        double ob = 0.0;
        if (l + 1 < m->n_layers) {
            for (int t : m->cross[l]) ob = ob + static_cast<double>(numel(m->tensors[t]) * static_cast<int64_t>(elt_bytes(m->tensors[t].dtype)));
        } else {
            const auto& t = m->tensors[m->layer_out[l]];
            ob = static_cast<double>(numel(t) * static_cast<int64_t>(elt_bytes(t.dtype)));
        }
        out[l].out_bytes = ob;
        out[l].rd_width = rdw;
        out[l].reserved = 0;
    }
    return MOPAR_OK;
}

// ---------------------------------------------------------------------------
// Validation and workspace layout
// ---------------------------------------------------------------------------

static int validate_and_build(mopar_model_s& m) {
    const int nt = static_cast<int>(m.tensors.size());
    const int epc = m.dtype == MOPAR_BF16 ? 8 : 4;       // channel granule of the GEMM loads
    const size_t es = elt_bytes(m.dtype);
    auto tid_ok = [&](int t) { return t >= 0 && t < nt; };
    if (!tid_ok(m.input) || !tid_ok(m.output) || m.input == m.output)
        return set_error(MOPAR_E_ARG, "model: bad input/output tensor id");
    for (int t = 0; t < nt; ++t) {
        const auto& d = m.tensors[t];
        if (d.rank < 1 || d.rank > 4) return set_error(MOPAR_E_SHAPE, "tensor " + std::to_string(t) + ": rank");
        for (int i = 0; i < d.rank; ++i)
            if (d.dims[i] < 1) return set_error(MOPAR_E_SHAPE, "tensor " + std::to_string(t) + ": dims must be >= 1");
        if (d.dtype != m.dtype && !(t == m.input && (d.dtype == MOPAR_F32 || d.dtype == MOPAR_I32)))
            return set_error(MOPAR_E_DTYPE, "tensor " + std::to_string(t) + ": dtype must be the model dtype");
    }
    std::vector<int> producer(nt, -1);
    std::vector<int64_t> filled(nt, 0);          // channels written so far by partial (concat) writers
    std::vector<int> last_writer(nt, -1);
    int prev_layer = -1;
    m.layer_first.assign(m.n_layers, -1);
    m.layer_last.assign(m.n_layers, -1);
    m.info.assign(m.ops.size(), OpInfo{});
    auto wcheck = [&](int64_t off, int64_t elems, const std::string& what) -> bool {
        if (off < 0 || off % 16 != 0) return false;
        const int64_t bytes = elems * static_cast<int64_t>(es);
        return static_cast<uint64_t>(off) + static_cast<uint64_t>(bytes) <= m.weights_bytes;
        (void)what;
    };
    for (int i = 0; i < static_cast<int>(m.ops.size()); ++i) {
        const auto& op = m.ops[i];
        auto& inf = m.info[i];
        const std::string nm = op_name(m, i);
        if (op.layer < 0 || op.layer >= m.n_layers || op.layer < prev_layer)
            return set_error(MOPAR_E_ARG, nm + ": layer index out of range or decreasing");
        if (op.layer != prev_layer) {
            if (op.layer != prev_layer + 1) return set_error(MOPAR_E_ARG, nm + ": a planning node has no ops");
            m.layer_first[op.layer] = i;
        }
        m.layer_last[op.layer] = i;
        prev_layer = op.layer;
        if (op.branch < 0 || (op.branch > 0 && op.pos < 1)) return set_error(MOPAR_E_ARG, nm + ": branch/pos");
        if (!tid_ok(op.in0) || !tid_ok(op.out) || (op.in1 != -1 && !tid_ok(op.in1)))
            return set_error(MOPAR_E_ARG, nm + ": tensor id out of range");
        // a conv whose output tensor is wider than n_out fills channels [out_off, out_off + n_out)
        const bool partial = op.kind == MOPAR_OP_CONV && m.tensors[op.out].rank == 4 &&
                             m.tensors[op.out].dims[1] > op.n_out;
        if (op.out == m.input) return set_error(MOPAR_E_ARG, nm + ": writes the model input");
        if (partial) {
            const auto& y = m.tensors[op.out];
            if (op.out_off != filled[op.out] || op.out_off + op.n_out > y.dims[1] || op.in1 >= 0)
                return set_error(MOPAR_E_ARG, nm + ": concatenating writers must fill the channels in order, "
                                                   "without overlap or residual");
            if (producer[op.out] != -1 && m.ops[producer[op.out]].layer != op.layer)
                return set_error(MOPAR_E_ARG, nm + ": concatenating writers of a tensor must share a node");
        } else {
            if (op.out_off != 0) return set_error(MOPAR_E_ARG, nm + ": out_off without a wider output tensor");
            if (producer[op.out] != -1) return set_error(MOPAR_E_ARG, nm + ": output tensor written twice");
        }
        for (int t : {op.in0, op.in1}) {
            if (t < 0) continue;
            if (t != m.input && producer[t] < 0)
                return set_error(MOPAR_E_ARG, nm + ": reads a tensor before it is produced");
            if (t != m.input && last_writer[t] >= 0 && filled[t] != m.tensors[t].dims[1])
                return set_error(MOPAR_E_ARG, nm + ": reads a concatenated tensor before all its channels are written");
            // single-input planning nodes: every op reads tensors of its own node, or the
            // tensor leaving the previous node (or the model input for node 0)
            if (t == m.input) {
                if (op.layer != 0) return set_error(MOPAR_E_ARG, nm + ": only node 0 may read the model input");
            } else {
                // tensors of its own node, or the output of any earlier node (skip edges
                // make a cut carry several tensors)
                const int pl = m.ops[producer[t]].layer;
                if (pl != op.layer && !(pl < op.layer && t == m.ops[m.layer_last[pl]].out))
                    return set_error(MOPAR_E_ARG, nm + ": reads a tensor that is neither its node's nor an earlier node's output");
            }
        }
        if (op.in1 >= 0 && op.kind != MOPAR_OP_CONV && op.kind != MOPAR_OP_LINEAR && op.kind != MOPAR_OP_LAYERNORM)
            return set_error(MOPAR_E_ARG, nm + ": second input only for conv, linear, layernorm");
        if (op.act < 0 || op.act > 2) return set_error(MOPAR_E_ARG, nm + ": act");
        if (op.rd && op.kind != MOPAR_OP_CONV && op.kind != MOPAR_OP_LINEAR)
            return set_error(MOPAR_E_ARG, nm + ": only conv and linear ops can be resource-dominant");
        const auto& x = m.tensors[op.in0];
        const auto& y = m.tensors[op.out];
        const bool xin = op.in0 == m.input;
        if (xin && x.dtype == MOPAR_I32 && op.kind != MOPAR_OP_EMBED && op.kind != MOPAR_OP_EMBED_BERT)
            return set_error(MOPAR_E_DTYPE, nm + ": token ids feed only embeddings");
        if (xin && x.dtype == MOPAR_F32 && m.dtype == MOPAR_BF16 && op.kind != MOPAR_OP_CONV)
            return set_error(MOPAR_E_UNSUPPORTED, nm + ": a float32 image input feeds only a conv");
        switch (op.kind) {
            case MOPAR_OP_CONV: {
                if (x.rank != 4 || op.kh < 1 || op.kw < 1 || op.stride < 1 || op.pad < 0 || op.n_out < 1)
                    return set_error(MOPAR_E_SHAPE, nm + ": conv geometry");
                const int64_t ho = (x.dims[2] + 2 * op.pad - op.kh) / op.stride + 1;
                const int64_t wo = (x.dims[3] + 2 * op.pad - op.kw) / op.stride + 1;
                if (ho < 1 || wo < 1 || !shape_eq(y, {x.dims[0], partial ? y.dims[1] : op.n_out, ho, wo}))
                    return set_error(MOPAR_E_SHAPE, nm + ": conv output shape");
                if (op.in1 >= 0 && !shape_eq(m.tensors[op.in1], {x.dims[0], op.n_out, ho, wo}))
                    return set_error(MOPAR_E_SHAPE, nm + ": residual shape");
                inf.input_is_model = xin;
                if (xin && x.dtype != MOPAR_F32) return set_error(MOPAR_E_DTYPE, nm + ": image input must be f32");
                if (!xin && x.dims[1] % epc != 0)
                    return set_error(MOPAR_E_UNSUPPORTED, nm + ": input channels must be a multiple of " +
                                                              std::to_string(epc));
                inf.cs = static_cast<int>(xin ? round_up(x.dims[1], epc) : x.dims[1]);
                inf.K = static_cast<int64_t>(op.kh) * op.kw * inf.cs;
                inf.M = x.dims[0] * ho * wo;
                if (!gemm_operands_fit(x.dims[0] * x.dims[2] * x.dims[3] * inf.cs * es, op.n_out * inf.K * es))
                    return set_error(MOPAR_E_UNSUPPORTED, nm + ": a GEMM operand reaches 2 GiB");
                if (!wcheck(op.w, op.n_out * inf.K, "w") || !wcheck(op.b, op.n_out, "b"))
                    return set_error(MOPAR_E_ARG, nm + ": weight offsets out of range or not 16-byte aligned");
                if (xin) inf.temps.push_back(static_cast<size_t>(x.dims[0] * x.dims[2] * x.dims[3] * inf.cs) * es);
                inf.splits = conv_halo_ok(m.dtype, op.kh, op.kw, op.stride, op.pad, inf.cs, op.n_out,
                                          static_cast<int>(ho), static_cast<int>(wo), inf.M)
                                 ? 1
                                 : gemm_splits(inf.M, op.n_out, static_cast<int>(inf.K), m.dtype, EPI_STD);
                if (inf.splits > 1) {
                    inf.partial_temp = static_cast<int>(inf.temps.size());
                    inf.temps.push_back(gemm_partial_bytes(inf.M, op.n_out, inf.splits));
                }
                break;
            }
            case MOPAR_OP_LINEAR: {
                const int64_t K = x.rank == 4 ? x.dims[1] * x.dims[2] * x.dims[3] : x.dims[x.rank - 1];
                const int64_t M = numel(x) / K;
                if (op.n_out < 1 || numel(y) != M * op.n_out || y.dims[y.rank - 1] != op.n_out)
                    return set_error(MOPAR_E_SHAPE, nm + ": linear output shape");
                if (x.rank != 4 && (y.rank != x.rank || !std::equal(x.dims, x.dims + x.rank - 1, y.dims)))
                    return set_error(MOPAR_E_SHAPE, nm + ": linear leading dims");
                if (op.in1 >= 0 && numel(m.tensors[op.in1]) != numel(y))
                    return set_error(MOPAR_E_SHAPE, nm + ": residual shape");
                if (K % epc != 0) return set_error(MOPAR_E_UNSUPPORTED, nm + ": K must be a multiple of " + std::to_string(epc));
                if (!gemm_operands_fit(M * K * es, op.n_out * K * es))
                    return set_error(MOPAR_E_UNSUPPORTED, nm + ": a GEMM operand reaches 2 GiB");
                inf.K = K;
                inf.M = M;
                if (!wcheck(op.w, op.n_out * K, "w") || !wcheck(op.b, op.n_out, "b"))
                    return set_error(MOPAR_E_ARG, nm + ": weight offsets out of range or not 16-byte aligned");
                inf.splits = gemm_splits(M, op.n_out, static_cast<int>(K), m.dtype, EPI_STD);
                if (inf.splits > 1) {
                    inf.partial_temp = static_cast<int>(inf.temps.size());
                    inf.temps.push_back(gemm_partial_bytes(M, op.n_out, inf.splits));
                }
                inf.ctr_temp = static_cast<int>(inf.temps.size());
                inf.temps.push_back(kWideCtrBytes);
                break;
            }
            case MOPAR_OP_MAXPOOL: {
                if (x.rank != 4 || op.kh < 1 || op.kh != op.kw || op.stride < 1 || op.pad < 0 || 2 * op.pad > op.kh)
                    return set_error(MOPAR_E_SHAPE, nm + ": pool geometry (square window, pad <= k/2)");
                const int64_t ho = (x.dims[2] + 2 * op.pad - op.kh) / op.stride + 1;
                const int64_t wo = (x.dims[3] + 2 * op.pad - op.kw) / op.stride + 1;
                if (!shape_eq(y, {x.dims[0], x.dims[1], ho, wo}))
                    return set_error(MOPAR_E_SHAPE, nm + ": pool output shape");
                if (x.dims[1] % epc != 0) return set_error(MOPAR_E_UNSUPPORTED, nm + ": channels granule");
                break;
            }
            case MOPAR_OP_AVGPOOL:
                if (x.rank != 4 || !shape_eq(y, {x.dims[0], x.dims[1]}))
                    return set_error(MOPAR_E_SHAPE, nm + ": avgpool shapes");
                break;
            case MOPAR_OP_LAYERNORM: {
                const int64_t f = x.dims[x.rank - 1];
                if (numel(y) != numel(x) || y.dims[y.rank - 1] != f) return set_error(MOPAR_E_SHAPE, nm + ": LN shapes");
                if (op.in1 >= 0 && numel(m.tensors[op.in1]) != numel(x)) return set_error(MOPAR_E_SHAPE, nm + ": LN residual");
                if (f > 2048) return set_error(MOPAR_E_UNSUPPORTED, nm + ": LN width > 2048");
                if (!wcheck(op.w, f, "g") || !wcheck(op.b, f, "b"))
                    return set_error(MOPAR_E_ARG, nm + ": weight offsets out of range or not 16-byte aligned");
                break;
            }
            case MOPAR_OP_ATTENTION: {
                if (x.rank != 3 || op.heads < 1 || x.dims[2] != 3 * 64 * static_cast<int64_t>(op.heads) ||
                    !shape_eq(y, {x.dims[0], x.dims[1], 64 * static_cast<int64_t>(op.heads)}))
                    return set_error(MOPAR_E_SHAPE, nm + ": attention needs (B,S,3*64*heads) -> (B,S,64*heads)");
                if (x.dims[1] > 128) return set_error(MOPAR_E_UNSUPPORTED, nm + ": attention seq > 128");
                break;
            }
            case MOPAR_OP_EMBED_BERT: {
                if (!xin || x.dtype != MOPAR_I32 || x.rank != 2 || y.rank != 3 || y.dims[0] != x.dims[0] ||
                    y.dims[1] != x.dims[1])
                    return set_error(MOPAR_E_SHAPE, nm + ": embedding needs ids (B,S) -> (B,S,F)");
                const int64_t f = y.dims[2];
                if (op.rows[0] < 1 || op.rows[1] < x.dims[1] || op.rows[2] < 1 || f > 2048)
                    return set_error(MOPAR_E_SHAPE, nm + ": table rows (positions must cover seq)");
                if (op.rows[0] >= (int64_t(1) << 31)) return set_error(MOPAR_E_UNSUPPORTED, nm + ": vocabulary >= 2^31");
                if (!wcheck(op.w, op.rows[0] * f, "tok") || !wcheck(op.w2, op.rows[1] * f, "pos") ||
                    !wcheck(op.w3, op.rows[2] * f, "type") || !wcheck(op.w4, f, "g") || !wcheck(op.w5, f, "b"))
                    return set_error(MOPAR_E_ARG, nm + ": weight offsets out of range or not 16-byte aligned");
                break;
            }
            case MOPAR_OP_EMBED: {
                if (!xin || x.dtype != MOPAR_I32 || y.rank != x.rank + 1 || y.dims[0] != x.dims[0])
                    return set_error(MOPAR_E_SHAPE, nm + ": embedding needs ids -> (..., F)");
                const int64_t f = y.dims[y.rank - 1];
                if ((f * static_cast<int64_t>(es)) % 16 != 0) return set_error(MOPAR_E_UNSUPPORTED, nm + ": row bytes % 16");
                if (op.rows[0] >= (int64_t(1) << 31)) return set_error(MOPAR_E_UNSUPPORTED, nm + ": vocabulary >= 2^31");
                if (op.rows[0] < 1 || !wcheck(op.w, op.rows[0] * f, "table"))
                    return set_error(MOPAR_E_ARG, nm + ": weight offsets out of range or not 16-byte aligned");
                break;
            }
            case MOPAR_OP_LSTM: {
                if (x.rank != 3 || op.n_out < 1 || !shape_eq(y, {x.dims[0], x.dims[1], op.n_out}))
                    return set_error(MOPAR_E_SHAPE, nm + ": LSTM (B,T,E) -> (B,T,H)");
                const int64_t e = x.dims[2], h = op.n_out;
                if (e % epc != 0 || h % epc != 0) return set_error(MOPAR_E_UNSUPPORTED, nm + ": E and H granule");
                if (!wcheck(op.w, 4 * h * e, "w_ih") || !wcheck(op.w2, 4 * h * h, "w_hh") || !wcheck(op.b, 4 * h, "b_ih") ||
                    !wcheck(op.w3, 4 * h, "b_hh"))
                    return set_error(MOPAR_E_ARG, nm + ": weight offsets out of range or not 16-byte aligned");
                const int64_t bt = x.dims[0] * x.dims[1];
                if (!gemm_operands_fit(bt * std::max(e, h) * es, 4 * h * std::max(e, h) * es))
                    return set_error(MOPAR_E_UNSUPPORTED, nm + ": a GEMM operand reaches 2 GiB");
                inf.temps.push_back(static_cast<size_t>(bt * 4 * h) * 4);       // input projection, f32
                inf.temps.push_back(static_cast<size_t>(x.dims[0] * h) * 4);    // cell state, f32
                if (lstm_recurrence_ok(m.dtype, x.dims[0], x.dims[1], h))       // one-launch recurrence:
                    inf.temps.push_back(lstm_recurrence_sync_bytes(x.dims[0], x.dims[1], h));   // step sync
                else
                    inf.temps.push_back(static_cast<size_t>(x.dims[0] * h) * es);   // h_0 = 0
                inf.ctr_temp = static_cast<int>(inf.temps.size());
                inf.temps.push_back(kWideCtrBytes);                               // input projection tiles
                break;
            }
            default: return set_error(MOPAR_E_ARG, nm + ": unknown op kind");
        }
        if (producer[op.out] == -1) producer[op.out] = i;
        if (partial) {
            filled[op.out] += op.n_out;
            last_writer[op.out] = i;
        }
    }
    for (int t = 0; t < nt; ++t)
        if (last_writer[t] >= 0 && filled[t] != m.tensors[t].dims[1])
            return set_error(MOPAR_E_ARG, "tensor " + std::to_string(t) + ": concatenating writers leave channels unwritten");
    if (prev_layer != m.n_layers - 1) return set_error(MOPAR_E_ARG, "model: a planning node has no ops");
    if (producer[m.output] != static_cast<int>(m.ops.size()) - 1)
        return set_error(MOPAR_E_ARG, "model: the output must be produced by the last op");
    m.layer_out.resize(m.n_layers);
    for (int l = 0; l < m.n_layers; ++l) m.layer_out[l] = m.ops[m.layer_last[l]].out;
    // tensors crossing each cut: produced as the output of a node <= j, read by a node > j
    m.cross.assign(m.n_layers > 1 ? m.n_layers - 1 : 0, {});
    {
        std::vector<int> last_reader_node(nt, -1), out_node(nt, -1);
        for (int l = 0; l < m.n_layers; ++l) out_node[m.layer_out[l]] = l;
        for (const auto& op : m.ops)
            for (int t : {op.in0, op.in1})
                if (t >= 0) last_reader_node[t] = std::max(last_reader_node[t], op.layer);
        for (int t = 0; t < nt; ++t)
            if (out_node[t] >= 0)
                for (int j = out_node[t]; j < last_reader_node[t] && j + 1 < m.n_layers; ++j) m.cross[j].push_back(t);
        for (int j = 0; j + 1 < m.n_layers; ++j)
            if (m.cross[j].empty()) return set_error(MOPAR_E_ARG, "model: nothing crosses the cut after node " + std::to_string(j));
    }

    // workspace: every tensor except the model input and output gets a slot, live from
    // its producer to its last reader; op scratch lives for its op.  First-fit reuse.
    std::vector<int> last_use(nt, -1);
    for (int i = 0; i < static_cast<int>(m.ops.size()); ++i)
        for (int t : {m.ops[i].in0, m.ops[i].in1})
            if (t >= 0) last_use[t] = i;
    struct Block { size_t off, size; int until; };
    std::vector<Block> live;
    size_t top = 0;
    auto alloc = [&](size_t bytes, int until) {
        bytes = (bytes + 255) / 256 * 256;
        std::sort(live.begin(), live.end(), [](const Block& a, const Block& b) { return a.off < b.off; });
        size_t cur = 0;
        for (const auto& b : live) {
            if (b.off >= cur + bytes) break;
            cur = std::max(cur, b.off + b.size);
        }
        live.push_back({cur, bytes, until});
        top = std::max(top, cur + bytes);
        return cur;
    };
    m.offset.assign(nt, SIZE_MAX);
    for (int i = 0; i < static_cast<int>(m.ops.size()); ++i) {
        live.erase(std::remove_if(live.begin(), live.end(), [&](const Block& b) { return b.until < i; }), live.end());
        auto& inf = m.info[i];
        inf.temp_off.clear();
        for (size_t tb : inf.temps) inf.temp_off.push_back(alloc(tb, i));
        const int t = m.ops[i].out;
        if (t != m.output && m.offset[t] == SIZE_MAX) {   // first writer allocates (concatenations)
            const size_t bytes = static_cast<size_t>(numel(m.tensors[t])) * es;
            m.offset[t] = alloc(bytes, std::max(last_use[t], i));
        }
    }
    m.ws_bytes = top;
    return MOPAR_OK;
}

int model_create_impl(const mopar_model_desc* d, const void* weights, size_t wbytes, mopar_model_t* out) {
    if (!d || !out) return set_error(MOPAR_E_ARG, "mopar_model_create: null argument");
    *out = nullptr;
    if (d->dtype != MOPAR_F32 && d->dtype != MOPAR_BF16)
        return set_error(MOPAR_E_DTYPE, "mopar_model_create: model dtype must be f32 or bf16");
    if (d->n_tensors < 2 || !d->tensors || d->n_ops < 1 || !d->ops || d->n_layers < 1)
        return set_error(MOPAR_E_ARG, "mopar_model_create: empty model");
    if (!weights && wbytes) return set_error(MOPAR_E_ARG, "mopar_model_create: null weights");
    auto* m = new mopar_model_s();
    m->dtype = d->dtype;
    m->tensors.assign(d->tensors, d->tensors + d->n_tensors);
    m->ops.assign(d->ops, d->ops + d->n_ops);
    m->n_layers = d->n_layers;
    m->input = d->input;
    m->output = d->output;
    m->weights = static_cast<const unsigned char*>(weights);
    m->weights_bytes = wbytes;
    const int rc = validate_and_build(*m);
    if (rc != MOPAR_OK) {
        delete m;
        return rc;
    }
    *out = m;
    return MOPAR_OK;
}

void model_destroy_impl(mopar_model_t m) { delete m; }

// ---------------------------------------------------------------------------
// Plans against a model
// ---------------------------------------------------------------------------

static int check_plan(const mopar_model_s* m, const mopar_plan* p, const char* who) {
    if (!m || !p || !p->slice_end || !p->k) return set_error(MOPAR_E_ARG, std::string(who) + ": null model or plan");
    if (p->n_layers != m->n_layers) return set_error(MOPAR_E_ARG, std::string(who) + ": plan is for another model");
    if (p->n_slices < 1 || p->n_slices > m->n_layers) return set_error(MOPAR_E_ARG, std::string(who) + ": n_slices");
    int prev = -1;
    for (int s = 0; s < p->n_slices; ++s) {
        if (p->slice_end[s] <= prev || p->slice_end[s] >= m->n_layers)
            return set_error(MOPAR_E_ARG, std::string(who) + ": slice_end must increase");
        prev = p->slice_end[s];
    }
    if (prev != m->n_layers - 1) return set_error(MOPAR_E_ARG, std::string(who) + ": last slice must end at the last node");
    for (int l = 0; l < m->n_layers; ++l) {
        int minw = 0;
        for (int i = m->layer_first[l]; i <= m->layer_last[l]; ++i)
            if (m->ops[i].rd) minw = minw == 0 ? m->ops[i].n_out : std::min(minw, m->ops[i].n_out);
        if (p->k[l] < 1 || (p->k[l] > 1 && (minw == 0 || p->k[l] > minw)))
            return set_error(MOPAR_E_ARG, std::string(who) + ": k[" + std::to_string(l) + "] invalid for that node");
    }
    return MOPAR_OK;
}

bool model_timing_enabled(const mopar_model_s* m) { return m && m->timing; }

int workspace_bytes_impl(const mopar_model_s* m, const mopar_plan* p, size_t* bytes) {
    if (!bytes) return set_error(MOPAR_E_ARG, "mopar_model_workspace_bytes: null output");
    const int rc = check_plan(m, p, "mopar_model_workspace_bytes");
    if (rc) return rc;
    *bytes = m->ws_bytes;
    return MOPAR_OK;
}

// ---------------------------------------------------------------------------
// Execution
// ---------------------------------------------------------------------------

struct Ptrs {
    const mopar_model_s* m;
    unsigned char* ws;
    const void* in_ptr;   // pointer bound to tensor in_tid
    int in_tid;
    void* out_ptr;        // pointer bound to tensor out_tid
    int out_tid;
    void* get(int t) const {
        if (t == in_tid) return const_cast<void*>(in_ptr);
        if (t == out_tid) return out_ptr;
        return ws + m->offset[t];
    }
};

static const void* W(const mopar_model_s& m, int64_t off) { return off < 0 ? nullptr : m.weights + off; }

static hipError_t run_op(const mopar_model_s& m, int i, const Ptrs& P, int ksub, hipStream_t s) {
    const auto& op = m.ops[i];
    const auto& inf = m.info[i];
    const auto& x = m.tensors[op.in0];
    const auto& y = m.tensors[op.out];
    const int dt = m.dtype;
    switch (op.kind) {
        case MOPAR_OP_CONV: {
            const void* src = P.get(op.in0);
            if (inf.input_is_model) {
                void* tmp = P.ws + inf.temp_off[0];
                hipError_t e = launch_nchw_to_nhwc(static_cast<const float*>(src), tmp, static_cast<int>(x.dims[0]),
                                                   static_cast<int>(x.dims[1]), static_cast<int>(x.dims[2]),
                                                   static_cast<int>(x.dims[3]), inf.cs, dt, s);
                if (e != hipSuccess) return e;
                src = tmp;
            }
            GemmParams g{};
            g.A = src;
            // a 1x1, stride-1, unpadded conv over channels-last pixels is a plain GEMM
            g.conv = (op.kh == 1 && op.kw == 1 && op.stride == 1 && op.pad == 0) ? 0 : 1;
            g.lda = inf.cs;
            g.img_h = static_cast<int>(x.dims[2]);
            g.img_w = static_cast<int>(x.dims[3]);
            g.cs = inf.cs;
            g.out_h = static_cast<int>(y.dims[2]);
            g.out_w = static_cast<int>(y.dims[3]);
            g.kh = op.kh;
            g.kw = op.kw;
            g.stride = op.stride;
            g.pad = op.pad;
            g.B = W(m, op.w);
            g.bias = W(m, op.b);
            g.res = op.in1 >= 0 ? P.get(op.in1) : nullptr;
            g.ldc = y.dims[1];                     // > n_out when the op fills part of a concatenation
            g.C = static_cast<unsigned char*>(P.get(op.out)) + static_cast<size_t>(op.out_off) * elt_bytes(m.dtype);
            g.M = inf.M;
            g.N = op.n_out;
            g.K = static_cast<int>(inf.K);
            g.act = op.act;
            g.ksub = ksub;
            g.splits = inf.splits;
            g.partial = inf.partial_temp >= 0 ? reinterpret_cast<float*>(P.ws + inf.temp_off[inf.partial_temp]) : nullptr;
            return launch_gemm(g, dt, s);
        }
        case MOPAR_OP_LINEAR: {
            GemmParams g{};
            g.A = P.get(op.in0);
            g.lda = inf.K;
            g.B = W(m, op.w);
            g.bias = W(m, op.b);
            g.res = op.in1 >= 0 ? P.get(op.in1) : nullptr;
            g.C = P.get(op.out);
            g.ldc = op.n_out;
            g.M = inf.M;
            g.N = op.n_out;
            g.K = static_cast<int>(inf.K);
            g.act = op.act;
            g.ksub = ksub;
            g.splits = inf.splits;
            g.partial = inf.partial_temp >= 0 ? reinterpret_cast<float*>(P.ws + inf.temp_off[inf.partial_temp]) : nullptr;
            g.wide_ctr = reinterpret_cast<unsigned*>(P.ws + inf.temp_off[inf.ctr_temp]);
            return launch_gemm(g, dt, s);
        }
        case MOPAR_OP_MAXPOOL:
            return launch_maxpool(P.get(op.in0), P.get(op.out), static_cast<int>(x.dims[0]), static_cast<int>(x.dims[2]),
                                  static_cast<int>(x.dims[3]), static_cast<int>(x.dims[1]), op.kh, op.stride, op.pad,
                                  static_cast<int>(y.dims[2]), static_cast<int>(y.dims[3]), dt, s);
        case MOPAR_OP_AVGPOOL:
            return launch_avgpool(P.get(op.in0), P.get(op.out), static_cast<int>(x.dims[0]),
                                  static_cast<int>(x.dims[2] * x.dims[3]), static_cast<int>(x.dims[1]), dt, s);
        case MOPAR_OP_LAYERNORM: {
            const int64_t f = x.dims[x.rank - 1];
            return launch_layernorm(P.get(op.in0), op.in1 >= 0 ? P.get(op.in1) : nullptr, W(m, op.w), W(m, op.b),
                                    P.get(op.out), numel(x) / f, static_cast<int>(f), op.eps, dt, s);
        }
        case MOPAR_OP_ATTENTION:
            return launch_attention(P.get(op.in0), P.get(op.out), static_cast<int>(x.dims[0]),
                                    static_cast<int>(x.dims[1]), op.heads, op.scale, dt, s);
        case MOPAR_OP_EMBED_BERT:
            return launch_embed_bert(static_cast<const int32_t*>(P.get(op.in0)), W(m, op.w), W(m, op.w2), W(m, op.w3),
                                     W(m, op.w4), W(m, op.w5), P.get(op.out), static_cast<int>(x.dims[0]),
                                     static_cast<int>(x.dims[1]), static_cast<int>(op.rows[0]),
                                     static_cast<int>(y.dims[2]), op.eps, dt, s);
        case MOPAR_OP_EMBED:
            return launch_embed(static_cast<const int32_t*>(P.get(op.in0)), W(m, op.w), P.get(op.out), numel(x),
                                static_cast<int>(y.dims[y.rank - 1]), static_cast<int>(op.rows[0]), dt, s);
        case MOPAR_OP_LSTM: {
            const int B = static_cast<int>(x.dims[0]), T = static_cast<int>(x.dims[1]), E = static_cast<int>(x.dims[2]);
            const int H = op.n_out;
            float* gx = reinterpret_cast<float*>(P.ws + inf.temp_off[0]);
            float* cst = reinterpret_cast<float*>(P.ws + inf.temp_off[1]);
            void* h0 = P.ws + inf.temp_off[2];
            const bool one_launch = lstm_recurrence_ok(dt, B, T, H);
            hipError_t e = hipSuccess;
            if (!one_launch) {
                e = launch_fill_zero(cst, static_cast<size_t>(B) * H * 4, s);
                if (e == hipSuccess) e = launch_fill_zero(h0, static_cast<size_t>(B) * H * dtype_size(dt), s);
                if (e != hipSuccess) return e;
            }
            // input projection for all steps: gx = x W_ih^T + b_ih + b_hh (float32)
            GemmParams g{};
            g.A = P.get(op.in0);
            g.lda = E;
            g.B = W(m, op.w);
            g.bias = W(m, op.b);
            g.bias2 = W(m, op.w3);
            g.C = gx;
            g.ldc = 4 * H;
            g.M = static_cast<int64_t>(B) * T;
            g.N = 4 * H;
            g.K = E;
            g.ksub = 1;
            g.out_f32 = 1;
            g.wide_ctr = reinterpret_cast<unsigned*>(P.ws + inf.temp_off[inf.ctr_temp]);
            e = launch_gemm(g, dt, s);
            if (e != hipSuccess) return e;
            if (one_launch) return launch_lstm_recurrence(gx, W(m, op.w2), P.get(op.out), cst, h0, B, T, H, s);
            // otherwise one GEMM per step with the cell update fused in its epilogue
            unsigned char* hseq = static_cast<unsigned char*>(P.get(op.out));
            const size_t es = dtype_size(dt);
            for (int t = 0; t < T; ++t) {
                GemmParams r{};
                r.A = t == 0 ? h0 : hseq + static_cast<size_t>(t - 1) * H * es;
                r.lda = t == 0 ? H : static_cast<int64_t>(T) * H;
                r.B = W(m, op.w2);
                r.C = hseq + static_cast<size_t>(t) * H * es;
                r.ldc = static_cast<int64_t>(T) * H;
                r.M = B;
                r.N = 4 * H;
                r.K = H;
                r.ksub = 1;
                r.epi = EPI_LSTM;
                r.gx = gx + static_cast<size_t>(t) * 4 * H;
                r.ldgx = static_cast<int64_t>(T) * 4 * H;
                r.cstate = cst;
                e = launch_gemm(r, dt, s);
                if (e != hipSuccess) return e;
            }
            return hipSuccess;
        }
        default: return hipErrorInvalidValue;
    }
}

// Runs `fn` (which enqueues work on s), bracketed by the events of `slot` when timing is on.
template <typename F>
static hipError_t timed(const mopar_model_s& mc, int slot, hipStream_t s, F&& fn) {
    auto& m = const_cast<mopar_model_s&>(mc);
    (void)s;
    if (!m.timing || slot < 0 || slot >= static_cast<int>(m.slot_lo.size())) return fn();
    LaunchTimer timer{&m.kev, &m.kev_next, hipSuccess};
    m.slot_lo[slot] = m.kev_next;
    t_timer = &timer;
    const hipError_t e = fn();
    t_timer = nullptr;
    m.slot_hi[slot] = m.kev_next;
    return e != hipSuccess ? e : timer.err;
}

static void reset_timing(const mopar_model_s& mc) {
    auto& m = const_cast<mopar_model_s&>(mc);
    m.kev_next = 0;
    std::fill(m.slot_lo.begin(), m.slot_lo.end(), 0);
    std::fill(m.slot_hi.begin(), m.slot_hi.end(), 0);
}

static int run_layers(const mopar_model_s& m, const mopar_plan& p, int l0, int l1, const Ptrs& P, hipStream_t s) {
    for (int l = l0; l <= l1; ++l)
        for (int i = m.layer_first[l]; i <= m.layer_last[l]; ++i) {
            const int ksub = m.ops[i].rd ? p.k[l] : 1;
            const hipError_t e = timed(m, i, s, [&] { return run_op(m, i, P, ksub, s); });
            if (e != hipSuccess) return hip_check(e, "kernel launch");
        }
    return MOPAR_OK;
}

int set_timing_impl(mopar_model_s* m, int32_t enable) {
    if (!m) return set_error(MOPAR_E_ARG, "mopar_model_set_timing: null model");
    m->free_events();
    const size_t n = m->ops.size() + 2 * static_cast<size_t>(m->n_layers - 1);
    m->timing = enable != 0;
    m->slot_lo.assign(enable ? n : 0, 0);
    m->slot_hi.assign(enable ? n : 0, 0);
    return MOPAR_OK;
}

int timing_slots_impl(const mopar_model_s* m, int32_t* n) {
    if (!m || !n) return set_error(MOPAR_E_ARG, "mopar_model_timing_slots: null argument");
    *n = static_cast<int32_t>(m->ops.size() + 2 * static_cast<size_t>(m->n_layers - 1));
    return MOPAR_OK;
}

int op_times_impl(const mopar_model_s* m, float* ms, int32_t n) {
    if (!m || !ms) return set_error(MOPAR_E_ARG, "mopar_model_op_times: null argument");
    if (!m->timing) return set_error(MOPAR_E_ARG, "mopar_model_op_times: timing is not enabled");
    for (int32_t i = 0; i < n; ++i) {
        ms[i] = -1.0f;
        if (i >= static_cast<int32_t>(m->slot_lo.size()) || m->slot_hi[i] <= m->slot_lo[i]) continue;
        float sum = 0.0f;
        for (size_t k = m->slot_lo[i]; k < m->slot_hi[i]; ++k) {
            int rc = hip_check(hipEventSynchronize(m->kev[k].second), "hipEventSynchronize");
            if (rc) return rc;
            float t = 0.0f;
            rc = hip_check(hipEventElapsedTime(&t, m->kev[k].first, m->kev[k].second), "hipEventElapsedTime");
            if (rc) return rc;
            sum += t;
        }
        ms[i] = sum;
    }
    return MOPAR_OK;
}

int slice_forward_impl(const mopar_model_s* m, const mopar_plan* p, int32_t s, const void* in, void* out, void* ws,
                       size_t ws_bytes, void* stream) {
    int rc = check_plan(m, p, "mopar_slice_forward");
    if (rc) return rc;
    if (s < 0 || s >= p->n_slices) return set_error(MOPAR_E_ARG, "mopar_slice_forward: slice index out of range");
    if (!in || !out) return set_error(MOPAR_E_ARG, "mopar_slice_forward: null input or output");
    if (m->ws_bytes && (!ws || ws_bytes < m->ws_bytes))
        return set_error(MOPAR_E_WORKSPACE, "mopar_slice_forward: workspace smaller than mopar_model_workspace_bytes");
    const int l0 = s == 0 ? 0 : p->slice_end[s - 1] + 1, l1 = p->slice_end[s];
    Ptrs P{m, static_cast<unsigned char*>(ws), in, s == 0 ? m->input : m->layer_out[l0 - 1], out, m->layer_out[l1]};
    reset_timing(*m);
    return run_layers(*m, *p, l0, l1, P, static_cast<hipStream_t>(stream));
}

// ---------------------------------------------------------------------------
// Measured layer profile: t_p(l, eta) for the parallelism search
// ---------------------------------------------------------------------------

int measure_impl(mopar_model_s* m, int32_t k_max, int32_t reps, const void* in, void* out, void* ws,
                 size_t ws_bytes, void* stream, double* tp) {
    if (!m || !in || !out || !tp) return set_error(MOPAR_E_ARG, "mopar_model_measure: null argument");
    if (k_max < 1 || k_max > 64 || reps < 1 || reps > 1000)
        return set_error(MOPAR_E_ARG, "mopar_model_measure: k_max must be 1..64 and reps 1..1000");
    if (m->ws_bytes && (!ws || ws_bytes < m->ws_bytes))
        return set_error(MOPAR_E_WORKSPACE, "mopar_model_measure: workspace smaller than mopar_model_workspace_bytes");
    const int n = m->n_layers;
    std::vector<int> minw(n, 0);                 // narrowest RD op of each node (0: none)
    for (int l = 0; l < n; ++l)
        for (int i = m->layer_first[l]; i <= m->layer_last[l]; ++i)
            if (m->ops[i].rd) minw[l] = minw[l] == 0 ? m->ops[i].n_out : std::min(minw[l], m->ops[i].n_out);
    const bool was_timing = m->timing;
    int rc = set_timing_impl(m, 1);
    if (rc) return rc;
    std::vector<int32_t> end{n - 1}, k(n, 1);
    mopar_plan plan{};
    plan.n_layers = n;
    plan.n_slices = 1;
    plan.slice_end = end.data();
    plan.k = k.data();
    const size_t nslot = m->ops.size() + 2 * static_cast<size_t>(n - 1);
    std::vector<float> ms(nslot);
    std::vector<std::vector<double>> samples(n);
    for (int eta = 1; eta <= k_max && !rc; ++eta) {
        for (int l = 0; l < n; ++l) k[l] = minw[l] ? std::min(eta, minw[l]) : 1;
        for (auto& v : samples) v.clear();
        for (int r = -1; r < reps && !rc; ++r) {   // r = -1: warm-up
            rc = slice_forward_impl(m, &plan, 0, in, out, ws, ws_bytes, stream);
            if (!rc) rc = op_times_impl(m, ms.data(), static_cast<int32_t>(nslot));
            if (rc || r < 0) continue;
            for (int l = 0; l < n; ++l) {
                double t = 0.0;
                for (int i = m->layer_first[l]; i <= m->layer_last[l]; ++i) t += ms[i] > 0.0f ? ms[i] : 0.0f;
                samples[l].push_back(t * 1e-3);
            }
        }
        if (rc) break;
        for (int l = 0; l < n; ++l) {
            auto v = samples[l];
            std::sort(v.begin(), v.end());
            tp[static_cast<size_t>(l) * k_max + eta - 1] = v[v.size() / 2];   // median (upper)
        }
    }
    const int rc2 = set_timing_impl(m, was_timing ? 1 : 0);
    return rc ? rc : rc2;
}

// ---------------------------------------------------------------------------
// Boundary codec
// ---------------------------------------------------------------------------

static int codec_geometry(const mopar_codec* c, const mopar_tensor_desc* x, int64_t* positions, int* channels,
                          const char* who) {
    if (!c || !x) return set_error(MOPAR_E_ARG, std::string(who) + ": null codec or descriptor");
    if (x->rank < 1 || x->rank > 4) return set_error(MOPAR_E_SHAPE, std::string(who) + ": rank");
    for (int i = 0; i < x->rank; ++i)
        if (x->dims[i] < 1) return set_error(MOPAR_E_SHAPE, std::string(who) + ": dims must be >= 1");
    if (x->dtype != MOPAR_F32 && x->dtype != MOPAR_BF16) return set_error(MOPAR_E_DTYPE, std::string(who) + ": dtype");
    const int64_t ch = x->rank == 4 ? x->dims[1] : x->dims[x->rank - 1];
    *channels = static_cast<int>(ch);
    *positions = numel(*x) / ch;
    if (c->kind == MOPAR_CODEC_RAW) return MOPAR_OK;
    if (c->kind != MOPAR_CODEC_AE) return set_error(MOPAR_E_ARG, std::string(who) + ": codec kind");
    if (c->c != ch) return set_error(MOPAR_E_SHAPE, std::string(who) + ": codec channels differ from the tensor's");
    if (c->c_code < 1) return set_error(MOPAR_E_ARG, std::string(who) + ": c_code must be >= 1");
    if (!c->w_enc || !c->w_dec) return set_error(MOPAR_E_ARG, std::string(who) + ": null codec weights");
    const int64_t es = elt_bytes(x->dtype);
    if (!gemm_operands_fit(*positions * std::max<int64_t>(ch, c->c_code) * es, int64_t(c->c_code) * ch * es))
        return set_error(MOPAR_E_UNSUPPORTED, std::string(who) + ": a codec GEMM operand reaches 2 GiB");
    return MOPAR_OK;
}

int code_bytes_impl(const mopar_codec* c, const mopar_tensor_desc* x, size_t* bytes) {
    int64_t pos;
    int ch;
    if (!bytes) return set_error(MOPAR_E_ARG, "mopar_boundary_code_bytes: null output");
    const int rc = codec_geometry(c, x, &pos, &ch, "mopar_boundary_code_bytes");
    if (rc) return rc;
    const int64_t per = c->kind == MOPAR_CODEC_RAW ? ch : c->c_code;
    *bytes = static_cast<size_t>(pos * per) * elt_bytes(x->dtype);
    return MOPAR_OK;
}

static hipError_t codec_apply(const mopar_codec& c, int dtype, int64_t pos, int ch, const void* src, void* dst,
                              bool encode, hipStream_t s) {
    if (c.kind == MOPAR_CODEC_RAW) return launch_copy(src, dst, static_cast<size_t>(pos * ch) * elt_bytes(dtype), s);
    // the layer's input width must sit on the GEMM's 16-byte granule; otherwise the vector-ALU kernel
    const int cin = encode ? c.c : c.c_code, cout = encode ? c.c_code : c.c;
    if (cin % (dtype == MOPAR_BF16 ? 8 : 4) != 0)
        return launch_codec_narrow(src, encode ? c.w_enc : c.w_dec, encode ? c.b_enc : c.b_dec, dst, pos, cin, cout,
                                   dtype, s);
    GemmParams g{};
    g.A = src;
    g.lda = encode ? c.c : c.c_code;
    g.B = encode ? c.w_enc : c.w_dec;
    g.bias = encode ? c.b_enc : c.b_dec;
    g.C = dst;
    g.ldc = encode ? c.c_code : c.c;
    g.M = pos;
    g.N = encode ? c.c_code : c.c;
    g.K = encode ? c.c : c.c_code;
    g.ksub = 1;
    g.thin = 1;
    return launch_gemm(g, dtype, s);
}

int encode_impl(const mopar_codec* c, const mopar_tensor_desc* x, const void* xd, void* code, void* stream) {
    int64_t pos;
    int ch;
    int rc = codec_geometry(c, x, &pos, &ch, "mopar_boundary_encode");
    if (rc) return rc;
    if (!xd || !code) return set_error(MOPAR_E_ARG, "mopar_boundary_encode: null device pointer");
    return hip_check(codec_apply(*c, x->dtype, pos, ch, xd, code, true, static_cast<hipStream_t>(stream)),
                     "mopar_boundary_encode");
}

int decode_impl(const mopar_codec* c, const mopar_tensor_desc* y, const void* code, void* yd, void* stream) {
    int64_t pos;
    int ch;
    int rc = codec_geometry(c, y, &pos, &ch, "mopar_boundary_decode");
    if (rc) return rc;
    if (!yd || !code) return set_error(MOPAR_E_ARG, "mopar_boundary_decode: null device pointer");
    return hip_check(codec_apply(*c, y->dtype, pos, ch, code, yd, false, static_cast<hipStream_t>(stream)),
                     "mopar_boundary_decode");
}

// ---------------------------------------------------------------------------
// Whole model
// ---------------------------------------------------------------------------

int model_forward_impl(const mopar_model_s* m, const mopar_plan* p, const mopar_codec* codecs, const void* in,
                       void* out, void* const* code_bufs, void* ws, size_t ws_bytes, void* stream) {
    int rc = check_plan(m, p, "mopar_model_forward");
    if (rc) return rc;
    if (!in || !out) return set_error(MOPAR_E_ARG, "mopar_model_forward: null input or output");
    if (m->ws_bytes && (!ws || ws_bytes < m->ws_bytes))
        return set_error(MOPAR_E_WORKSPACE, "mopar_model_forward: workspace smaller than mopar_model_workspace_bytes");
    const int S = p->n_slices;
    if (S > 1 && (!codecs || !code_bufs)) return set_error(MOPAR_E_ARG, "mopar_model_forward: codecs / code buffers");
    // boundary b: the tensors crossing cut 0, then cut 1, ... (ascending tensor id within a cut);
    // validate every codec against its tensor before enqueuing anything
    std::vector<int> base(S, 0);
    for (int s = 0; s + 1 < S; ++s) {
        const auto& cr = m->cross[p->slice_end[s]];
        base[s + 1] = base[s] + static_cast<int>(cr.size());
        for (size_t q = 0; q < cr.size(); ++q) {
            int64_t pos;
            int ch;
            rc = codec_geometry(&codecs[base[s] + q], &m->tensors[cr[q]], &pos, &ch, "mopar_model_forward");
            if (rc) return rc;
            if (!code_bufs[base[s] + q]) return set_error(MOPAR_E_ARG, "mopar_model_forward: null code buffer");
        }
    }
    const hipStream_t st = static_cast<hipStream_t>(stream);
    Ptrs P{m, static_cast<unsigned char*>(ws), in, m->input, out, m->output};
    reset_timing(*m);
    const int slot0 = static_cast<int>(m->ops.size());
    // encode (to = true) or decode every tensor crossing the cut after slice c
    auto hand_off = [&](int c, bool enc) -> hipError_t {
        const auto& cr = m->cross[p->slice_end[c]];
        for (size_t q = 0; q < cr.size(); ++q) {
            const auto& t = m->tensors[cr[q]];
            const int b = base[c] + static_cast<int>(q);
            int64_t pos;
            int ch;
            codec_geometry(&codecs[b], &t, &pos, &ch, "mopar_model_forward");
            const hipError_t e = enc ? codec_apply(codecs[b], t.dtype, pos, ch, P.get(cr[q]), code_bufs[b], true, st)
                                     : codec_apply(codecs[b], t.dtype, pos, ch, code_bufs[b], P.get(cr[q]), false, st);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    };
    int l0 = 0;
    for (int s = 0; s < S; ++s) {
        const int l1 = p->slice_end[s];
        if (s > 0) {   // decode the previous boundary into this slice's inputs
            rc = hip_check(timed(*m, slot0 + 2 * (s - 1) + 1, st, [&] { return hand_off(s - 1, false); }),
                           "boundary decode");
            if (rc) return rc;
        }
        rc = run_layers(*m, *p, l0, l1, P, st);
        if (rc) return rc;
        if (s + 1 < S) {   // encode this slice's outputs into the boundary buffers
            rc = hip_check(timed(*m, slot0 + 2 * s, st, [&] { return hand_off(s, true); }), "boundary encode");
            if (rc) return rc;
        }
        l0 = l1 + 1;
    }
    return MOPAR_OK;
}

int cut_tensors_impl(const mopar_model_s* m, int32_t node, int32_t* tids, int32_t cap, int32_t* count) {
    if (!m || !count || (cap > 0 && !tids)) return set_error(MOPAR_E_ARG, "mopar_model_cut_tensors: null argument");
    if (node < 0 || node + 1 >= m->n_layers) return set_error(MOPAR_E_ARG, "mopar_model_cut_tensors: node out of range");
    const auto& cr = m->cross[node];
    *count = static_cast<int32_t>(cr.size());
    for (int32_t i = 0; i < cap && i < *count; ++i) tids[i] = cr[i];
    return MOPAR_OK;
}

}  // namespace mopar

// ---------------------------------------------------------------------------
// Slice pipeline across requests
// ---------------------------------------------------------------------------

struct mopar_pipeline_s {
    const mopar_model_s* m = nullptr;
    std::vector<int32_t> slice_end, k;
    mopar_plan plan{};
    std::vector<mopar_codec> codecs;
    int S = 0, depth = 0, replicas = 0;
    std::vector<hipStream_t> streams;              // [replicas][S]
    std::vector<unsigned char*> ws;                // [replicas][S], one model workspace each
    std::vector<int> base;                         // first boundary tensor of each cut
    int nb = 0;                                    // boundary tensors over all cuts
    std::vector<void*> codes;                      // [replicas][depth][nb]
    std::vector<hipEvent_t> enc_done, dec_done;    // [replicas][depth][S-1]
    int64_t submitted = 0;
    // graph replay: one executable graph per (ring slot, input, output), captured on first use
    bool graphs = false;
    struct Graph {
        int slot;
        const void* in;
        void* out;
        hipGraphExec_t exec;
    };
    std::vector<Graph> gexec;
    void drop_graphs() {
        for (auto& g : gexec) (void)hipGraphExecDestroy(g.exec);
        gexec.clear();
    }
    ~mopar_pipeline_s() {
        drop_graphs();
        for (auto e : enc_done) (void)hipEventDestroy(e);
        for (auto e : dec_done) (void)hipEventDestroy(e);
    }
};

namespace mopar {

static size_t slice_ws_stride(const mopar_model_s* m) { return (m->ws_bytes + 255) / 256 * 256; }

int pipeline_ws_bytes_impl(const mopar_model_s* m, const mopar_plan* p, int32_t replicas, size_t* bytes) {
    if (!bytes) return set_error(MOPAR_E_ARG, "mopar_pipeline_workspace_bytes: null output");
    if (replicas < 1 || replicas > 64) return set_error(MOPAR_E_ARG, "mopar_pipeline_workspace_bytes: replicas 1..64");
    const int rc = check_plan(m, p, "mopar_pipeline_workspace_bytes");
    if (rc) return rc;
    *bytes = slice_ws_stride(m) * static_cast<size_t>(p->n_slices) * static_cast<size_t>(replicas);
    return MOPAR_OK;
}

int pipeline_create_impl(const mopar_model_s* m, const mopar_plan* p, const mopar_codec* codecs, int32_t replicas,
                         int32_t depth, void* const* streams, void* ws, size_t ws_bytes, void* const* code_bufs,
                         mopar_pipeline_t* out) {
    if (!out) return set_error(MOPAR_E_ARG, "mopar_pipeline_create: null output");
    *out = nullptr;
    int rc = check_plan(m, p, "mopar_pipeline_create");
    if (rc) return rc;
    const int S = p->n_slices;
    if (depth < 1 || depth > 64) return set_error(MOPAR_E_ARG, "mopar_pipeline_create: depth must be 1..64");
    if (replicas < 1 || replicas > 64) return set_error(MOPAR_E_ARG, "mopar_pipeline_create: replicas must be 1..64");
    if (!streams) return set_error(MOPAR_E_ARG, "mopar_pipeline_create: null streams");
    const size_t need = slice_ws_stride(m) * static_cast<size_t>(S) * static_cast<size_t>(replicas);
    if (need && (!ws || ws_bytes < need))
        return set_error(MOPAR_E_WORKSPACE, "mopar_pipeline_create: workspace smaller than mopar_pipeline_workspace_bytes");
    if (S > 1 && (!codecs || !code_bufs)) return set_error(MOPAR_E_ARG, "mopar_pipeline_create: codecs / code buffers");
    std::vector<int> base(S > 1 ? S - 1 : 0, 0);
    int nb = 0;
    for (int c = 0; c + 1 < S; ++c) {
        base[c] = nb;
        nb += static_cast<int>(m->cross[p->slice_end[c]].size());
    }
    for (int c = 0; c + 1 < S; ++c) {
        const auto& cr = m->cross[p->slice_end[c]];
        for (size_t q = 0; q < cr.size(); ++q) {
            int64_t pos;
            int ch;
            rc = codec_geometry(&codecs[base[c] + q], &m->tensors[cr[q]], &pos, &ch, "mopar_pipeline_create");
            if (rc) return rc;
            for (int r = 0; r < replicas * depth; ++r)
                if (!code_bufs[r * nb + base[c] + q]) return set_error(MOPAR_E_ARG, "mopar_pipeline_create: null code buffer");
        }
    }
    auto* pp = new mopar_pipeline_s();
    pp->m = m;
    pp->slice_end.assign(p->slice_end, p->slice_end + S);
    pp->k.assign(p->k, p->k + m->n_layers);
    pp->plan = *p;
    pp->plan.slice_end = pp->slice_end.data();
    pp->plan.k = pp->k.data();
    if (S > 1) pp->codecs.assign(codecs, codecs + nb);
    pp->base = base;
    pp->nb = nb;
    pp->S = S;
    pp->depth = depth;
    pp->replicas = replicas;
    for (int i = 0; i < replicas * S; ++i) {
        pp->streams.push_back(static_cast<hipStream_t>(streams[i]));
        pp->ws.push_back(static_cast<unsigned char*>(ws) + slice_ws_stride(m) * static_cast<size_t>(i));
    }
    const int ncut = S - 1;
    for (int i = 0; i < replicas * depth * nb; ++i) pp->codes.push_back(code_bufs[i]);
    for (int i = 0; i < replicas * depth * ncut; ++i) {
        hipEvent_t a, b;
        rc = hip_check(hipEventCreateWithFlags(&a, hipEventDisableTiming), "hipEventCreateWithFlags");
        if (rc) {
            delete pp;
            return rc;
        }
        rc = hip_check(hipEventCreateWithFlags(&b, hipEventDisableTiming), "hipEventCreateWithFlags");
        if (rc) {
            (void)hipEventDestroy(a);
            delete pp;
            return rc;
        }
        pp->enc_done.push_back(a);
        pp->dec_done.push_back(b);
    }
    *out = pp;
    return MOPAR_OK;
}

// Enqueue batch `in` -> `out` on instance `rep`, ring slot `r`.  `events` = false leaves out the
// cross-stream events: valid when the instance runs all its slices on one stream, whose order
// then already puts slice s after slice s-1 and a slot's encode after its previous decode.
static int enqueue_batch(mopar_pipeline_s* pp, int rep, int r, const void* in, void* out, bool events) {
    const mopar_model_s& m = *pp->m;
    const int S = pp->S, ncut = S - 1;
    int l0 = 0;
    for (int s = 0; s < S; ++s) {
        const int l1 = pp->slice_end[s];
        const hipStream_t st = pp->streams[rep * S + s];
        // slice s reads its input from the caller (s = 0) or from its own workspace (decoded)
        Ptrs P{&m, pp->ws[rep * S + s], in, s == 0 ? m.input : -1, out, s == S - 1 ? m.output : -1};
        int rc;
        // encode / decode every tensor crossing cut c with its own codec and ring buffer
        auto hand_off = [&](int c, bool enc) -> hipError_t {
            const auto& cr = m.cross[pp->slice_end[c]];
            for (size_t q = 0; q < cr.size(); ++q) {
                const auto& t = m.tensors[cr[q]];
                const int b = pp->base[c] + static_cast<int>(q);
                int64_t pos;
                int ch;
                codec_geometry(&pp->codecs[b], &t, &pos, &ch, "mopar_pipeline_submit");
                void* code = pp->codes[static_cast<size_t>(r) * pp->nb + b];
                const hipError_t e = enc ? codec_apply(pp->codecs[b], t.dtype, pos, ch, P.get(cr[q]), code, true, st)
                                         : codec_apply(pp->codecs[b], t.dtype, pos, ch, code, P.get(cr[q]), false, st);
                if (e != hipSuccess) return e;
            }
            return hipSuccess;
        };
        if (s > 0) {
            const int c = s - 1, slot = r * ncut + c;
            if (events) {
                rc = hip_check(hipStreamWaitEvent(st, pp->enc_done[slot], 0), "hipStreamWaitEvent");
                if (rc) return rc;
            }
            rc = hip_check(hand_off(c, false), "boundary decode");
            if (rc) return rc;
            if (events) {
                rc = hip_check(hipEventRecord(pp->dec_done[slot], st), "hipEventRecord");
                if (rc) return rc;
            }
        }
        for (int l = l0; l <= l1; ++l)
            for (int i = m.layer_first[l]; i <= m.layer_last[l]; ++i) {
                const int ksub = m.ops[i].rd ? pp->k[l] : 1;
                rc = hip_check(run_op(m, i, P, ksub, st), "kernel launch");
                if (rc) return rc;
            }
        if (s < S - 1) {
            const int c = s, slot = r * ncut + c;
            // the slot is free once the previous batch using it has been decoded
            if (events) {
                rc = hip_check(hipStreamWaitEvent(st, pp->dec_done[slot], 0), "hipStreamWaitEvent");
                if (rc) return rc;
            }
            rc = hip_check(hand_off(c, true), "boundary encode");
            if (rc) return rc;
            if (events) {
                rc = hip_check(hipEventRecord(pp->enc_done[slot], st), "hipEventRecord");
                if (rc) return rc;
            }
        }
        l0 = l1 + 1;
    }
    return MOPAR_OK;
}

int pipeline_submit_impl(mopar_pipeline_s* pp, const void* in, void* out) {
    if (!pp) return set_error(MOPAR_E_ARG, "mopar_pipeline_submit: null pipeline");
    if (!in || !out) return set_error(MOPAR_E_ARG, "mopar_pipeline_submit: null input or output");
    const int rep = static_cast<int>(pp->submitted % pp->replicas);               // instance
    const int r = static_cast<int>((pp->submitted / pp->replicas) % pp->depth) + rep * pp->depth;  // ring slot
    if (!pp->graphs) {
        const int rc = enqueue_batch(pp, rep, r, in, out, true);
        if (rc) return rc;
        ++pp->submitted;
        return MOPAR_OK;
    }
    const hipStream_t st = pp->streams[rep * pp->S];
    hipGraphExec_t exec = nullptr;
    for (const auto& g : pp->gexec)
        if (g.slot == r && g.in == in && g.out == out) exec = g.exec;
    if (!exec) {
        // capture the batch's kernels once; nothing reaches the GPU until the launch below
        int rc = hip_check(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
        if (rc) return rc;
        rc = enqueue_batch(pp, rep, r, in, out, false);
        hipGraph_t graph = nullptr;
        const hipError_t e = hipStreamEndCapture(st, &graph);
        if (rc == MOPAR_OK) rc = hip_check(e, "hipStreamEndCapture");
        if (rc == MOPAR_OK) rc = hip_check(hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0), "hipGraphInstantiate");
        if (graph) (void)hipGraphDestroy(graph);
        if (rc) return rc;
        pp->gexec.push_back({r, in, out, exec});
    }
    const int rc = hip_check(hipGraphLaunch(exec, st), "hipGraphLaunch");
    if (rc) return rc;
    ++pp->submitted;
    return MOPAR_OK;
}

int pipeline_use_graphs_impl(mopar_pipeline_s* pp, int32_t enable) {
    if (!pp) return set_error(MOPAR_E_ARG, "mopar_pipeline_use_graphs: null pipeline");
    if (enable) {
        for (int rep = 0; rep < pp->replicas; ++rep)
            for (int s = 1; s < pp->S; ++s)
                if (pp->streams[rep * pp->S + s] != pp->streams[rep * pp->S])
                    return set_error(MOPAR_E_UNSUPPORTED,
                                     "mopar_pipeline_use_graphs: an instance runs its slices on several streams");
    } else {
        pp->drop_graphs();
    }
    pp->graphs = enable != 0;
    return MOPAR_OK;
}

void pipeline_destroy_impl(mopar_pipeline_s* pp) { delete pp; }

}  // namespace mopar
