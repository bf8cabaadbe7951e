// Structure compilation and batch lowering; see plan.hpp.
#include "plan.hpp"

#include <algorithm>
#include <functional>
#include <map>
#include <mutex>
#include <utility>

namespace kgq {

// Models whose projection is an MLP pass per hop and that define negation
// (BetaE, ConE, LogicE); GQE and Query2Box translate, and fuse projection
// runs into chains.
static bool per_hop_mlp(int model) { return model == KGQ_BETAE || model == KGQ_CONE || model == KGQ_LOGICE; }

// ---------------------------------------------------------------------------
// Built-in structures
// ---------------------------------------------------------------------------

// The 14 query shapes of the benchmark the paper evaluates (Introduction;
// Experiments, Datasets & Tasks), in Table 1's column order, written as
// graphs. Slots are consumed in the order written; pin negates the one-hop
// branch, pni the two-hop branch; up projects a union, which the compiler
// distributes over the two branches (Eq. 1).
static const char* const kBuiltinText[kNumStructures] = {
    "p(e0,r0)",                          // 1p
    "p(p(e0,r0),r1)",                    // 2p
    "p(p(p(e0,r0),r1),r2)",              // 3p
    "i(p(e0,r0),p(e1,r1))",              // 2i
    "i(p(e0,r0),p(e1,r1),p(e2,r2))",     // 3i
    "i(p(p(e0,r0),r1),p(e1,r2))",        // pi
    "p(i(p(e0,r0),p(e1,r1)),r2)",        // ip
    "u(p(e0,r0),p(e1,r1))",              // 2u
    "p(u(p(e0,r0),p(e1,r1)),r2)",        // up
    "i(p(e0,r0),n(p(e1,r1)))",           // 2in
    "i(p(e0,r0),p(e1,r1),n(p(e2,r2)))",  // 3in
    "p(i(p(e0,r0),n(p(e1,r1))),r2)",     // inp
    "i(p(p(e0,r0),r1),n(p(e1,r2)))",     // pin
    "i(n(p(p(e0,r0),r1)),p(e1,r2))",     // pni
};
static const char* const kBuiltinName[kNumStructures] = {"1p", "2p",  "3p",  "2i",  "3i",  "pi",  "ip",
                                                         "2u", "up",  "2in", "3in", "inp", "pin", "pni"};

const char* builtin_text(int id) { return (id >= 0 && id < kNumStructures) ? kBuiltinText[id] : nullptr; }

// ---------------------------------------------------------------------------
// Text form
// ---------------------------------------------------------------------------

namespace {

kgq_node make_node(int op, int slot)
{
    kgq_node n;
    n.op = op;
    n.slot = slot;
    for (int j = 0; j < 4; ++j) n.in[j] = -1;
    return n;
}

struct Parser {
    const char* s;
    size_t pos;
    std::vector<kgq_node>& out;
    std::string& err;

    void ws()
    {
        while (s[pos] == ' ' || s[pos] == '\t' || s[pos] == '\n' || s[pos] == '\r') ++pos;
    }
    int fail(const std::string& m)
    {
        if (err.empty()) err = m + " at offset " + std::to_string(pos);
        return -1;
    }
    bool expect(char c)
    {
        ws();
        if (s[pos] != c) {
            fail(std::string("expected '") + c + "'");
            return false;
        }
        ++pos;
        return true;
    }
    bool number(int& v)
    {
        ws();
        if (s[pos] < '0' || s[pos] > '9') {
            fail("expected a slot number");
            return false;
        }
        long x = 0;
        while (s[pos] >= '0' && s[pos] <= '9') {
            x = x * 10 + (s[pos] - '0');
            if (x > 1000000) {
                fail("slot number too large");
                return false;
            }
            ++pos;
        }
        v = (int)x;
        return true;
    }
    int push(const kgq_node& n)
    {
        if ((int)out.size() >= kMaxGraphNodes) return fail("more than " + std::to_string(kMaxGraphNodes) + " nodes");
        out.push_back(n);
        return (int)out.size() - 1;
    }
    int expr(int depth)
    {
        if (depth > kMaxGraphNodes) return fail("nesting deeper than the node limit");
        ws();
        const char c = s[pos];
        if (c == 'e') {
            ++pos;
            int k = 0;
            if (!number(k)) return -1;
            return push(make_node(KGQ_OP_ANCHOR, k));
        }
        if (c == 'p') {
            ++pos;
            if (!expect('(')) return -1;
            const int x = expr(depth + 1);
            if (x < 0 || !expect(',')) return -1;
            ws();
            if (s[pos] != 'r') return fail("expected a relation slot r<k>");
            ++pos;
            int k = 0;
            if (!number(k) || !expect(')')) return -1;
            kgq_node n = make_node(KGQ_OP_PROJECT, k);
            n.in[0] = x;
            return push(n);
        }
        if (c == 'n') {
            ++pos;
            if (!expect('(')) return -1;
            const int x = expr(depth + 1);
            if (x < 0 || !expect(')')) return -1;
            kgq_node n = make_node(KGQ_OP_NOT, -1);
            n.in[0] = x;
            return push(n);
        }
        if (c == 'i' || c == 'u') {
            ++pos;
            if (!expect('(')) return -1;
            int ins[5];
            int k = 0;
            for (;;) {
                const int x = expr(depth + 1);
                if (x < 0) return -1;
                if (k == 4) return fail("an intersection or union takes at most 4 subqueries");
                ins[k++] = x;
                ws();
                if (s[pos] == ',') {
                    ++pos;
                    continue;
                }
                break;
            }
            if (!expect(')')) return -1;
            if (k < 2) return fail("an intersection or union takes at least 2 subqueries");
            kgq_node n = make_node(c == 'i' ? KGQ_OP_AND : KGQ_OP_OR, -1);
            for (int j = 0; j < k; ++j) n.in[j] = ins[j];
            return push(n);
        }
        return fail(c ? std::string("unexpected '") + c + "'" : std::string("unexpected end of text"));
    }
};

}  // namespace

bool parse_graph(const char* text, std::vector<kgq_node>& out, std::string& err)
{
    out.clear();
    err.clear();
    if (!text) {
        err = "text is NULL";
        return false;
    }
    Parser P{text, 0, out, err};
    if (P.expr(0) < 0) return false;
    P.ws();
    if (text[P.pos] != '\0') {
        P.fail("trailing characters");
        return false;
    }
    return true;
}

// ---------------------------------------------------------------------------
// Compilation: validation, normal form, fusion, schedule
// ---------------------------------------------------------------------------

namespace {

// A node of the normal-form graph: no unions; negations explicit.
struct IrNode {
    int op;        // KGQ_OP_ANCHOR, KGQ_OP_PROJECT, KGQ_OP_AND, KGQ_OP_NOT
    int slot;
    int n_in;
    int in[kMaxBranches];
};

constexpr size_t kMaxIrNodes = 4096;

int popcount(unsigned m)
{
    int c = 0;
    for (; m; m &= m - 1) ++c;
    return c;
}

}  // namespace

bool compile_graph(int model, const kgq_node* nodes, int n, const std::string& name, Program& P, std::string& err,
                   int& st)
{
    P = Program();
    P.name = name;
    auto bad = [&](const std::string& m) {
        err = (name.empty() ? std::string() : "structure " + name + ": ") + m;
        st = KGQ_E_INVALID_ARG;
        return false;
    };
    if (!nodes) return bad("nodes is NULL");
    if (n < 1 || n > kMaxGraphNodes) return bad("a graph has 1 to " + std::to_string(kMaxGraphNodes) + " nodes");

    // 1. Validate the captured graph.
    std::vector<int> uses(n, 0);
    unsigned amask = 0, rmask = 0;
    bool negation = false;
    for (int i = 0; i < n; ++i) {
        const kgq_node& x = nodes[i];
        const std::string at = "node " + std::to_string(i) + ": ";
        int k = 0;
        while (k < 4 && x.in[k] >= 0) ++k;
        for (int j = k; j < 4; ++j)
            if (x.in[j] != -1) return bad(at + "inputs must fill in[] from the front, unused entries -1");
        for (int j = 0; j < k; ++j)
            if (x.in[j] >= i) return bad(at + "an input must be an earlier node");
        switch (x.op) {
        case KGQ_OP_ANCHOR:
            if (k != 0) return bad(at + "an anchor takes no input");
            if (x.slot < 0 || x.slot >= kMaxSlots) return bad(at + "anchor slot outside [0, 8)");
            amask |= 1u << x.slot;
            break;
        case KGQ_OP_PROJECT:
            if (k != 1) return bad(at + "a projection takes one input");
            if (x.slot < 0 || x.slot >= kMaxSlots) return bad(at + "relation slot outside [0, 8)");
            rmask |= 1u << x.slot;
            break;
        case KGQ_OP_NOT:
            if (k != 1) return bad(at + "a negation takes one input");
            negation = true;
            break;
        case KGQ_OP_AND:
        case KGQ_OP_OR:
            if (k < 2) return bad(at + "an intersection or union takes 2 to 4 inputs");
            break;
        default: return bad(at + "unknown op " + std::to_string(x.op));
        }
        for (int j = 0; j < k; ++j) {
            ++uses[x.in[j]];
            if (nodes[x.in[j]].op == KGQ_OP_ANCHOR && x.op != KGQ_OP_PROJECT)
                return bad(at + "an anchor can only feed a projection");
        }
    }
    for (int i = 0; i + 1 < n; ++i)
        if (!uses[i]) return bad("node " + std::to_string(i) + " is not used (the answer is the last node)");
    if (nodes[n - 1].op == KGQ_OP_ANCHOR) return bad("the answer must not be an anchor");
    if ((amask & (amask + 1)) || (rmask & (rmask + 1)))
        return bad("anchor and relation slots must be numbered 0, 1, ... without gaps");
    if (negation && !per_hop_mlp(model)) {
        err = (name.empty() ? std::string() : "structure " + name + ": ") +
              "negation is defined for BetaE, ConE and LogicE only";
        st = KGQ_E_UNSUPPORTED;
        return false;
    }
    P.negation = negation;
    P.n_anchors = popcount(amask);
    P.n_relations = popcount(rmask);

    // 2. Disjunctive normal form (Eq. 1): the value of every node becomes a
    // list of conjunctive terms. A projection maps each term; an
    // intersection takes one term from each input in every combination (the
    // first input varying slowest); a union concatenates; the negation of
    // several terms is the intersection of their negations.
    std::vector<IrNode> ir;
    ir.reserve(64);
    auto add = [&](int op, int slot, std::initializer_list<int> ins) {
        IrNode x{op, slot, 0, {-1, -1, -1, -1}};
        for (int v : ins) x.in[x.n_in++] = v;
        ir.push_back(x);
        return (int)ir.size() - 1;
    };
    std::vector<std::vector<int>> terms(n);
    for (int i = 0; i < n; ++i) {
        const kgq_node& x = nodes[i];
        std::vector<int>& T = terms[i];
        int k = 0;
        while (k < 4 && x.in[k] >= 0) ++k;
        switch (x.op) {
        case KGQ_OP_ANCHOR: T.push_back(add(KGQ_OP_ANCHOR, x.slot, {})); break;
        case KGQ_OP_PROJECT:
            for (int t : terms[x.in[0]]) T.push_back(add(KGQ_OP_PROJECT, x.slot, {t}));
            break;
        case KGQ_OP_OR:
            for (int j = 0; j < k; ++j) T.insert(T.end(), terms[x.in[j]].begin(), terms[x.in[j]].end());
            break;
        case KGQ_OP_AND: {
            size_t total = 1;
            for (int j = 0; j < k; ++j) total *= terms[x.in[j]].size();
            if (total > (size_t)kMaxTerms) break;   // reported below
            for (size_t t = 0; t < total; ++t) {
                IrNode a{KGQ_OP_AND, -1, k, {-1, -1, -1, -1}};
                size_t rest = t;
                for (int j = k - 1; j >= 0; --j) {
                    const std::vector<int>& tj = terms[x.in[j]];
                    a.in[j] = tj[rest % tj.size()];
                    rest /= tj.size();
                }
                ir.push_back(a);
                T.push_back((int)ir.size() - 1);
            }
            break;
        }
        case KGQ_OP_NOT: {
            const std::vector<int>& ti = terms[x.in[0]];
            if (ti.size() == 1) {
                T.push_back(add(KGQ_OP_NOT, -1, {ti[0]}));
            } else {
                IrNode a{KGQ_OP_AND, -1, (int)ti.size(), {-1, -1, -1, -1}};
                for (size_t t = 0; t < ti.size(); ++t) a.in[t] = add(KGQ_OP_NOT, -1, {ti[t]});
                ir.push_back(a);
                T.push_back((int)ir.size() - 1);
            }
            break;
        }
        }
        if (T.empty() || T.size() > (size_t)kMaxTerms)
            return bad("node " + std::to_string(i) + " has more than " + std::to_string(kMaxTerms) +
                       " conjunctive terms in disjunctive normal form");
        if (ir.size() > kMaxIrNodes) return bad("the graph is too large once unions are distributed");
    }

    // 3. Fusion. Every use of a normal-form node becomes its own fused
    // operator (a tree), so that each operator has one consumer and its row
    // can be placed where that consumer reads it.
    std::vector<FusedOp>& ops = P.ops;
    bool too_many = false;
    auto push = [&](FusedOp&& f) {
        if ((int)ops.size() >= kMaxFusedOps) too_many = true;
        ops.push_back(std::move(f));
        return (int)ops.size() - 1;
    };
    std::function<int(int, bool&)> emit = [&](int id, bool& neg) -> int {
        const IrNode x = ir[id];
        if (x.op == KGQ_OP_NOT) {
            const int o = emit(x.in[0], neg);
            neg = !neg;
            return o;
        }
        if (x.op == KGQ_OP_AND) {
            FusedOp f;
            f.kind = OP_AND;
            for (int j = 0; j < x.n_in; ++j) {
                bool nj = false;
                const int o = emit(x.in[j], nj);
                f.in.push_back(o);
                f.in_neg.push_back(nj ? 1 : 0);
            }
            neg = false;
            return push(std::move(f));
        }
        // A maximal run of projections down to its source (horizontal).
        std::vector<int> rels;
        int cur = id;
        while (ir[cur].op == KGQ_OP_PROJECT) {
            rels.push_back(ir[cur].slot);
            cur = ir[cur].in[0];
        }
        std::reverse(rels.begin(), rels.end());
        int src = -1, anchor = -1;
        bool src_neg = false;
        if (ir[cur].op == KGQ_OP_ANCHOR) anchor = ir[cur].slot;
        else src = emit(cur, src_neg);
        neg = false;
        if (!per_hop_mlp(model)) {
            if (src < 0) {
                FusedOp f;
                f.kind = OP_CHAIN;
                f.anchor = anchor;
                f.rels = rels;
                return push(std::move(f));
            }
            // hybrid: the run continues the intersection that produced its
            // source (no negation on these models, so the source is an AND)
            ops[src].rels.insert(ops[src].rels.end(), rels.begin(), rels.end());
            return src;
        }
        int prev = src;
        for (size_t h = 0; h < rels.size(); ++h) {
            FusedOp f;
            f.kind = OP_PROJ;
            f.src = prev;
            f.anchor = prev < 0 ? anchor : -1;
            f.src_neg = h == 0 && src_neg;
            f.rels = {rels[h]};
            prev = push(std::move(f));
        }
        return prev;
    };
    for (int t : terms[n - 1]) {
        bool neg = false;
        const int o = emit(t, neg);
        P.answer.push_back(o);
        P.answer_neg.push_back(neg ? 1 : 0);
    }
    if (too_many) return bad("more than " + std::to_string(kMaxFusedOps) + " fused operators");
    P.n_terms = (int)P.answer.size();
    if (P.n_terms == 3) {   // groups of four scored rows; the max is unchanged by a repeat
        P.answer.push_back(P.answer.back());
        P.answer_neg.push_back(P.answer_neg.back());
    }

    // 4. Schedule positions (ops are created after their inputs).
    for (FusedOp& f : ops) {
        if (f.kind == OP_CHAIN) {
            f.stage = 0;
        } else if (f.kind == OP_PROJ) {
            f.stage = f.src < 0 ? 0 : ops[f.src].stage;
            f.hop = (f.src >= 0 && ops[f.src].kind == OP_PROJ) ? ops[f.src].hop + 1 : 1;
        } else {
            int s = 0;
            for (int o : f.in) s = std::max(s, ops[o].stage);
            f.stage = s + 1;
            P.and_stages = std::max(P.and_stages, f.stage);
        }
    }

    // 5. Per-query needs.
    std::map<std::pair<int, int>, int> level;
    std::map<int, int> st_in, st_groups;
    int words = 2 * (int)P.answer.size() + 1 + 2;   // score rows, output, arity
    for (const FusedOp& f : ops) {
        if (f.kind == OP_CHAIN) {
            words += 3 + (int)f.rels.size();
        } else if (f.kind == OP_PROJ) {
            words += 5;
            P.max_stage_level = std::max(P.max_stage_level, ++level[{f.stage, f.hop}]);
        } else {
            words += 5 + (int)f.rels.size();
            P.max_stage_inputs = std::max(P.max_stage_inputs, st_in[f.stage] += (int)f.in.size());
            P.max_stage_groups = std::max(P.max_stage_groups, ++st_groups[f.stage]);
        }
    }
    P.image_words = words;
    return true;
}

const Program* builtin_program(int model, int id)
{
    static std::vector<Program> table[5];
    static std::once_flag once;
    std::call_once(once, [] {
        for (int m = 0; m < 5; ++m) {
            table[m].resize(kNumStructures);
            for (int s = 0; s < kNumStructures; ++s) {
                std::vector<kgq_node> nodes;
                std::string err;
                int st = 0;
                parse_graph(kBuiltinText[s], nodes, err);
                if (!compile_graph(m, nodes.data(), (int)nodes.size(), kBuiltinName[s], table[m][s], err, st)) {
                    // negation structures on GQE / Query2Box: kept for their
                    // arity and name, rejected when a batch uses them
                    Program& P = table[m][s];
                    P = Program();
                    P.name = kBuiltinName[s];
                    P.supported = false;
                    P.negation = true;
                    Program full;
                    compile_graph(KGQ_BETAE, nodes.data(), (int)nodes.size(), kBuiltinName[s], full, err, st);
                    P.n_anchors = full.n_anchors;
                    P.n_relations = full.n_relations;
                }
            }
        }
    });
    if (model < 0 || model > 4 || id < 0 || id >= kNumStructures) return nullptr;
    return &table[model][id];
}

// ---------------------------------------------------------------------------
// Launch counts
// ---------------------------------------------------------------------------

// launches per intersection stage: dense layers + combines (LogicE: the
// t-norm combine only)
static int and_stage_launches(int model)
{
    switch (model) {
    case KGQ_GQE: return 3;
    case KGQ_Q2B: return 6;
    case KGQ_BETAE: return 4;
    case KGQ_CONE: return 6;
    default: return 1;
    }
}

// launches per projection level: (table gather | prep + layer 1) + layers 2,
// 3, and LogicE's bound map
static int level_launches(int model, bool table) { return (table ? 3 : 4) + (model == KGQ_LOGICE ? 1 : 0); }

int plan_launches(const Plan& p, bool topk)
{
    int n = 0;
    for (const Stage& s : p.stages) {
        if (s.kind == ST_CHAIN) n += 1;                                   // chains
        else if (s.kind == ST_LEVEL) n += level_launches(p.model, s.table);
        else n += and_stage_launches(p.model);
    }
    return n + 2 + (topk ? 1 : 0);                            // pack, score, top-k
}

int program_launches(int model, const Program& prog, bool topk)
{
    int n = prog.and_stages * and_stage_launches(model);
    if (per_hop_mlp(model)) {
        std::map<std::pair<int, int>, int> level;
        for (const FusedOp& f : prog.ops)
            if (f.kind == OP_PROJ) level[{f.stage, f.hop}] = 1;
        for (auto& kv : level) n += level_launches(model, kv.first.first == 0 && kv.first.second == 1);
    } else {
        for (const FusedOp& f : prog.ops)
            if (f.kind == OP_CHAIN) {
                n += 1;
                break;
            }
    }
    return n + 2 + (topk ? 1 : 0);
}

// ---------------------------------------------------------------------------
// Batch lowering
// ---------------------------------------------------------------------------

bool lower(int model, int B, const int32_t* sid, int fixed_sid, int a_stride, int r_stride, bool mixed,
           const std::vector<const Program*>& table, Plan& p, std::string& err, int& err_status)
{
    p = Plan();
    p.model = model;
    p.B = B;
    std::vector<const Program*> pq(B);
    int K = 0;
    for (int q = 0; q < B; ++q) {
        const int s = mixed ? sid[q] : fixed_sid;
        const Program* g = (s >= 0 && s < (int)table.size()) ? table[s] : nullptr;
        const std::string at = "query " + std::to_string(q) + ": ";
        if (!g) {
            err = at + "unknown structure id " + std::to_string(s);
            err_status = KGQ_E_INVALID_ARG;
            return false;
        }
        if (!g->supported) {
            err = at + "structure " + g->name + " uses negation, which this model does not define";
            err_status = KGQ_E_UNSUPPORTED;
            return false;
        }
        if (g->n_anchors > a_stride || g->n_relations > r_stride) {
            err = at + "structure " + g->name + " takes " + std::to_string(g->n_anchors) + " anchors and " +
                  std::to_string(g->n_relations) + " relations; this call holds " + std::to_string(a_stride) +
                  " and " + std::to_string(r_stride) + " per query";
            err_status = KGQ_E_INVALID_ARG;
            return false;
        }
        pq[q] = g;
        K = std::max(K, g->and_stages);
    }

    // Fused-operator instances: query q's op o is instance base[q] + o.
    std::vector<int64_t> base(B + 1, 0);
    for (int q = 0; q < B; ++q) base[q + 1] = base[q] + (int64_t)pq[q]->ops.size();
    std::vector<int32_t> row((size_t)base[B], -1);
    int next = 0;

    // Rows. Each intersection stage reads one contiguous block (its dense
    // layers run over the block), each group's inputs contiguous inside it;
    // the producers of those inputs write straight into the block. Every
    // other fused operator gets a row of its own.
    struct Grp { int q, op, start; };
    std::vector<std::vector<Grp>> grp(K + 1);
    std::vector<int> in_base(K + 1, 0), in_count(K + 1, 0);
    for (int k = 1; k <= K; ++k) {
        in_base[k] = next;
        for (int q = 0; q < B; ++q) {
            const std::vector<FusedOp>& ops = pq[q]->ops;
            for (int o = 0; o < (int)ops.size(); ++o) {
                if (ops[o].kind != OP_AND || ops[o].stage != k) continue;
                grp[k].push_back({q, o, next - in_base[k]});
                for (int i : ops[o].in) row[base[q] + i] = next++;
            }
        }
        in_count[k] = next - in_base[k];
    }
    for (auto& r : row)
        if (r < 0) r = next++;
    p.n_state_rows = next;

    auto put = [&](const std::vector<int32_t>& v) {
        const int64_t o = (int64_t)p.image.size();
        p.image.insert(p.image.end(), v.begin(), v.end());
        while (p.image.size() % 4) p.image.push_back(0);   // 16-byte aligned lists
        return o;
    };

    // GQE / Query2Box: every chain of the batch in one stage.
    if (!per_hop_mlp(model)) {
        std::vector<int32_t> aref, roff{0}, rref, dst;
        for (int q = 0; q < B; ++q) {
            const std::vector<FusedOp>& ops = pq[q]->ops;
            for (int o = 0; o < (int)ops.size(); ++o) {
                if (ops[o].kind != OP_CHAIN) continue;
                aref.push_back(q * a_stride + ops[o].anchor);
                for (int r : ops[o].rels) rref.push_back(q * r_stride + r);
                roff.push_back((int32_t)rref.size());
                dst.push_back(row[base[q] + o]);
            }
        }
        if (!aref.empty()) {
            Stage s;
            s.kind = ST_CHAIN;
            s.count = (int)aref.size();
            s.a = put(aref);
            s.b = put(roff);
            s.c = put(rref);
            s.d = put(dst);
            p.stages.push_back(s);
            p.n_anchor_chains = s.count;
        }
    }

    // MLP projections (BetaE, ConE, LogicE), bucketed by (stage, hop) in query order.
    std::map<std::pair<int, int>, std::vector<std::pair<int, int>>> levels;
    if (per_hop_mlp(model))
        for (int q = 0; q < B; ++q) {
            const std::vector<FusedOp>& ops = pq[q]->ops;
            for (int o = 0; o < (int)ops.size(); ++o)
                if (ops[o].kind == OP_PROJ) levels[{ops[o].stage, ops[o].hop}].push_back({q, o});
        }
    auto emit_levels = [&](int k) {
        for (auto it = levels.lower_bound({k, 0}); it != levels.end() && it->first.first == k; ++it) {
            std::vector<int32_t> src, aref, rref, neg, dst;
            for (auto& qo : it->second) {
                const int q = qo.first;
                const FusedOp& f = pq[q]->ops[qo.second];
                src.push_back(f.src >= 0 ? row[base[q] + f.src] : -1);
                aref.push_back(f.src < 0 ? q * a_stride + f.anchor : 0);
                rref.push_back(q * r_stride + f.rels[0]);
                neg.push_back(f.src_neg ? 1 : 0);
                dst.push_back(row[base[q] + qo.second]);
            }
            Stage s;
            s.kind = ST_LEVEL;
            s.stage = k;
            s.hop = it->first.second;
            s.count = (int)src.size();
            s.table = k == 0 && s.hop == 1;   // sources are anchors, never negated
            s.a = put(src);
            s.b = put(aref);
            s.c = put(rref);
            s.d = put(neg);
            s.e = put(dst);
            p.stages.push_back(s);
            p.level_rows[k > 0 ? 3 : std::min(s.hop, 3) - 1] += s.count;
            if (s.table) p.n_anchor_chains = s.count;
            p.max_level = std::max(p.max_level, s.count);
        }
    };
    auto emit_and = [&](int k) {
        if (grp[k].empty()) return;
        std::vector<int32_t> start, nin, out, mask, poff{0}, pref;
        for (const Grp& g : grp[k]) {
            const FusedOp& f = pq[g.q]->ops[g.op];
            start.push_back(g.start);
            nin.push_back((int32_t)f.in.size());
            out.push_back(row[base[g.q] + g.op]);
            int m = 0;
            for (size_t j = 0; j < f.in_neg.size(); ++j)
                if (f.in_neg[j]) m |= 1 << j;
            mask.push_back(m);
            for (int r : f.rels) pref.push_back(g.q * r_stride + r);
            poff.push_back((int32_t)pref.size());
        }
        Stage s;
        s.kind = ST_AND;
        s.stage = k;
        s.count = (int)start.size();
        s.in_base = in_base[k];
        s.n_in = in_count[k];
        s.a = put(start);
        s.b = put(nin);
        s.c = put(out);
        s.d = put(mask);
        s.e = put(poff);
        s.f = put(pref);
        p.stages.push_back(s);
        p.n_groups += s.count;
        p.n_int_in += s.n_in;
        p.n_and_stages += 1;
        p.max_and_in = std::max(p.max_and_in, s.n_in);
        p.max_and_groups = std::max(p.max_and_groups, s.count);
    };
    if (per_hop_mlp(model)) emit_levels(0);
    for (int k = 1; k <= K; ++k) {
        emit_and(k);
        if (per_hop_mlp(model)) emit_levels(k);
    }

    // Scored rows: groups of four, then pairs, then single rows.
    std::vector<int32_t> ssrc, sneg, odst;
    for (int width : {4, 2, 1}) {
        for (int q = 0; q < B; ++q) {
            const Program* g = pq[q];
            if ((int)g->answer.size() != width) continue;
            for (int t = 0; t < width; ++t) {
                ssrc.push_back(row[base[q] + g->answer[t]]);
                sneg.push_back(g->answer_neg[t]);
            }
            odst.push_back(q);
        }
        if (width == 4) p.n_quad_rows = (int)ssrc.size();
        if (width == 2) p.n_pair_rows = (int)ssrc.size() - p.n_quad_rows;
    }
    p.n_score_rows = (int)ssrc.size();
    p.off_score_src = put(ssrc);
    p.off_score_neg = put(sneg);
    p.off_out_dest = put(odst);
    if (mixed) {
        std::vector<int32_t> ar((size_t)2 * B);
        for (int q = 0; q < B; ++q) {
            ar[2 * q] = pq[q]->n_anchors;
            ar[2 * q + 1] = pq[q]->n_relations;
        }
        p.off_arity = put(ar);
    }
    return true;
}

}  // namespace kgq
