// Plan lowering for the 14 query structures; see plan.hpp.
#include "plan.hpp"

#include "../../include/kgq.h"

namespace kgq {

// Structure table. Shapes follow the standard 14-structure benchmark the
// paper evaluates (Introduction; Experiments, Datasets & Tasks); the union
// structures are written in disjunctive normal form (Eq. 1), so "up" pushes
// its final relation into both branches.
static const StructureDef kStructs[kNumStructures] = {
    // name  na nr nbr  branches                                                       merge      post neg
    {"1p", 1, 1, 1, {{0, 1, {0, -1, -1}, false}}, MERGE_NONE, -1, false},
    {"2p", 1, 2, 1, {{0, 2, {0, 1, -1}, false}}, MERGE_NONE, -1, false},
    {"3p", 1, 3, 1, {{0, 3, {0, 1, 2}, false}}, MERGE_NONE, -1, false},
    {"2i", 2, 2, 2, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, false}}, MERGE_AND, -1, false},
    {"3i", 3, 3, 3, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, false}, {2, 1, {2, -1, -1}, false}},
     MERGE_AND, -1, false},
    {"pi", 2, 3, 2, {{0, 2, {0, 1, -1}, false}, {1, 1, {2, -1, -1}, false}}, MERGE_AND, -1, false},
    {"ip", 2, 3, 2, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, false}}, MERGE_AND, 2, false},
    {"2u", 2, 2, 2, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, false}}, MERGE_OR, -1, false},
    {"up", 2, 3, 2, {{0, 2, {0, 2, -1}, false}, {1, 2, {1, 2, -1}, false}}, MERGE_OR, -1, false},
    {"2in", 2, 2, 2, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, true}}, MERGE_AND, -1, true},
    {"3in", 3, 3, 3, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, false}, {2, 1, {2, -1, -1}, true}},
     MERGE_AND, -1, true},
    {"inp", 2, 3, 2, {{0, 1, {0, -1, -1}, false}, {1, 1, {1, -1, -1}, true}}, MERGE_AND, 2, true},
    {"pin", 2, 3, 2, {{0, 2, {0, 1, -1}, false}, {1, 1, {2, -1, -1}, true}}, MERGE_AND, -1, true},
    {"pni", 2, 3, 2, {{0, 2, {0, 1, -1}, true}, {1, 1, {2, -1, -1}, false}}, MERGE_AND, -1, true},
};

const StructureDef* structure_def(int id)
{
    if (id < 0 || id >= kNumStructures) return nullptr;
    return &kStructs[id];
}

int64_t plan_image_words(int B)
{
    // chains 3B*(1+3); groups 5B; levels 4 * 3B * 4; scores 2B + B; arity 2B
    return (int64_t)B * (12 + 5 + 48 + 3 + 2) + 256;   // + per-section alignment padding
}

int plan_launches(const Plan& p, bool topk)
{
    int n = 0;
    if (p.model == KGQ_BETAE) {
        // first hop: table gather (first layer) + 2 dense layers; later
        // levels: prep + 3 dense layers
        for (int l = 0; l < 4; ++l)
            if (!p.lv_dst[l].empty()) n += (l == 0) ? 3 : 4;
        if (p.n_groups) n += 4;                         // prep, 2 dense layers, combine
    } else {
        n += 1;                                         // chains
        if (p.n_groups) n += (p.model == KGQ_Q2B) ? 6 : 3;
    }
    n += 2;                                             // pack + score
    if (topk) n += 1;
    return n;
}

bool lower(int model, int B, const int32_t* sid, int fixed_sid, int a_stride, int r_stride,
           bool mixed, Plan& p, std::string& err, int& err_status)
{
    p = Plan();
    p.model = model;
    p.B = B;
    std::vector<const StructureDef*> defs(B);
    for (int q = 0; q < B; ++q) {
        const int s = mixed ? sid[q] : fixed_sid;
        const StructureDef* d = structure_def(s);
        if (!d) {
            err = "query " + std::to_string(q) + ": unknown structure id " + std::to_string(s);
            err_status = KGQ_E_INVALID_ARG;
            return false;
        }
        if (d->negation && model != KGQ_BETAE) {
            err = "query " + std::to_string(q) + ": structure " + d->name +
                  " uses negation, which this model does not define";
            err_status = KGQ_E_UNSUPPORTED;
            return false;
        }
        defs[q] = d;
    }

    // Row regions: A intersection inputs, B union branches, C single chains.
    std::vector<int> and_q, or_q, none_q;
    for (int q = 0; q < B; ++q) {
        const int m = defs[q]->merge;
        (m == MERGE_AND ? and_q : m == MERGE_OR ? or_q : none_q).push_back(q);
    }
    struct ChainSrc { int q; const BranchDef* b; };
    std::vector<ChainSrc> chains;
    std::vector<int> chain_of_none(B, -1);
    for (int q : and_q) {
        p.g_in_start.push_back((int32_t)chains.size());
        p.g_n.push_back(defs[q]->n_branches);
        int neg = 0;
        for (int j = 0; j < defs[q]->n_branches; ++j) {
            if (defs[q]->br[j].negated) neg |= 1 << j;
            chains.push_back({q, &defs[q]->br[j]});
        }
        p.g_neg.push_back(neg);
    }
    p.n_int_in = (int)chains.size();
    std::vector<int> union_row0;
    for (int q : or_q) {
        union_row0.push_back((int)chains.size());
        for (int j = 0; j < 2; ++j) chains.push_back({q, &defs[q]->br[j]});
    }
    for (int q : none_q) {
        chain_of_none[q] = (int)chains.size();
        chains.push_back({q, &defs[q]->br[0]});
    }
    p.n_chain = (int)chains.size();
    p.n_groups = (int)and_q.size();
    int next_row = p.n_chain;

    // group outputs (region D)
    std::vector<int> scored_row_of_q(B, -1);
    for (int g = 0; g < p.n_groups; ++g) {
        const int q = and_q[g];
        p.g_out.push_back(next_row);
        scored_row_of_q[q] = next_row;
        ++next_row;
        const int post = defs[q]->post_rel;
        // GQE / Q2B fuse the post projection into the combine; BetaE runs it
        // as one more MLP level.
        p.g_post.push_back((model != KGQ_BETAE && post >= 0) ? q * r_stride + post : -1);
    }
    for (int q : none_q) scored_row_of_q[q] = chain_of_none[q];

    // chains: anchor / relation references into the caller's arrays
    p.chain_anchor_ref.resize(p.n_chain);
    p.chain_rel_ref.assign((size_t)p.n_chain * 3, -1);
    for (int c = 0; c < p.n_chain; ++c) {
        const int q = chains[c].q;
        const BranchDef* b = chains[c].b;
        p.chain_anchor_ref[c] = q * a_stride + b->anchor;
        for (int h = 0; h < b->n_hops; ++h) p.chain_rel_ref[(size_t)c * 3 + h] = q * r_stride + b->rel[h];
    }

    if (model == KGQ_BETAE) {
        // hop levels; intermediate hops get rows of their own (region F)
        std::vector<int> prev(p.n_chain, -1);
        for (int lvl = 0; lvl < 3; ++lvl) {
            for (int c = 0; c < p.n_chain; ++c) {
                const BranchDef* b = chains[c].b;
                if (lvl >= b->n_hops) continue;
                const int dst = (lvl == b->n_hops - 1) ? c : next_row++;
                p.lv_src[lvl].push_back(lvl == 0 ? -1 : prev[c]);
                p.lv_anchor[lvl].push_back(p.chain_anchor_ref[c]);
                p.lv_rel[lvl].push_back(p.chain_rel_ref[(size_t)c * 3 + lvl]);
                p.lv_dst[lvl].push_back(dst);
                prev[c] = dst;
            }
        }
        for (int g = 0; g < p.n_groups; ++g) {
            const int q = and_q[g];
            const int post = defs[q]->post_rel;
            if (post < 0) continue;
            p.lv_src[3].push_back(p.g_out[g]);
            p.lv_anchor[3].push_back(q * a_stride);
            p.lv_rel[3].push_back(q * r_stride + post);
            p.lv_dst[3].push_back(next_row);
            scored_row_of_q[q] = next_row++;
        }
    }
    p.n_state_rows = next_row;

    // scored rows: union pairs first (adjacent rows, pair-aligned), then the
    // other queries in input order
    for (size_t u = 0; u < or_q.size(); ++u) {
        p.score_src.push_back(union_row0[u]);
        p.score_src.push_back(union_row0[u] + 1);
        p.out_dest.push_back(or_q[u]);
    }
    p.n_union_rows = (int)p.score_src.size();
    for (int q = 0; q < B; ++q) {
        if (defs[q]->merge == MERGE_OR) continue;
        p.score_src.push_back(scored_row_of_q[q]);
        p.out_dest.push_back(q);
    }
    p.n_score_rows = (int)p.score_src.size();
    if (mixed) {
        p.arity.resize((size_t)2 * B);
        for (int q = 0; q < B; ++q) {
            p.arity[2 * q] = defs[q]->n_anchors;
            p.arity[2 * q + 1] = defs[q]->n_relations;
        }
    }

    // flatten
    auto put = [&](const std::vector<int32_t>& v) {
        const int64_t o = (int64_t)p.image.size();
        p.image.insert(p.image.end(), v.begin(), v.end());
        while (p.image.size() % 4) p.image.push_back(0);   // 16-byte aligned sections
        return o;
    };
    p.off.chain_anchor = put(p.chain_anchor_ref);
    p.off.chain_rel = put(p.chain_rel_ref);
    p.off.g_in_start = put(p.g_in_start);
    p.off.g_n = put(p.g_n);
    p.off.g_out = put(p.g_out);
    p.off.g_post = put(p.g_post);
    p.off.g_neg = put(p.g_neg);
    for (int l = 0; l < 4; ++l) {
        p.off.lv_src[l] = put(p.lv_src[l]);
        p.off.lv_anchor[l] = put(p.lv_anchor[l]);
        p.off.lv_rel[l] = put(p.lv_rel[l]);
        p.off.lv_dst[l] = put(p.lv_dst[l]);
    }
    p.off.score_src = put(p.score_src);
    p.off.out_dest = put(p.out_dest);
    p.off.arity = put(p.arity);
    return true;
}

}  // namespace kgq
