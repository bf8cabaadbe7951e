// Host driver for a sanitizer build (AddressSanitizer + UndefinedBehaviorSanitizer,
// g++ only: no device code) of the library's structure compiler: the text reader,
// the normal form and fusion (compile_graph) and the batch lowering (lower).
//
// usage: plan_driver <texts file> <seed>
// Every line of the file is a structure in text form, well formed or not. Each
// line is read; a graph that parses is compiled for all five models; a graph
// that compiles is lowered alone and inside mixed batches with the built-in
// structures, at several batch sizes and slot strides. Then random node arrays
// (out-of-range ops, slots and inputs included) go straight to compile_graph.
// Any memory error or undefined behaviour aborts the run (the sanitizers are
// built non-recovering); the driver itself only counts outcomes.
#include <cstdio>
#include <fstream>
#include <random>
#include <string>
#include <vector>

#include "../../paper_2503_02172_amd/csrc/plan.hpp"

using namespace kgq;

int main(int argc, char** argv)
{
    if (argc < 3) {
        std::fprintf(stderr, "usage: %s <texts> <seed>\n", argv[0]);
        return 2;
    }
    std::mt19937 rng((unsigned)std::stoul(argv[2]));
    std::ifstream in(argv[1]);
    std::string line;
    long parsed = 0, rejected = 0, compiled = 0, lowered = 0, lower_refused = 0;
    while (std::getline(in, line)) {
        std::vector<kgq_node> nodes;
        std::string err;
        if (!parse_graph(line.c_str(), nodes, err)) {
            ++rejected;
            continue;
        }
        ++parsed;
        for (int model = 0; model < 5; ++model) {
            Program P;
            int st = 0;
            if (!compile_graph(model, nodes.data(), (int)nodes.size(), "t", P, err, st)) continue;
            ++compiled;
            std::vector<const Program*> table;
            for (int id = 0; id < kNumStructures; ++id) table.push_back(builtin_program(model, id));
            table.push_back(&P);
            const int self = (int)table.size() - 1;
            (void)program_launches(model, P, true);
            for (int B : {1, 7, 64}) {
                Plan plan;
                int es = 0;
                const int sa = P.n_anchors > 0 ? P.n_anchors : 1, sr = P.n_relations > 0 ? P.n_relations : 1;
                if (lower(model, B, nullptr, self, sa, sr, false, table, plan, err, es)) {
                    ++lowered;
                    (void)plan_launches(plan, true);
                } else {
                    ++lower_refused;
                }
                // mixed: random structure ids, out-of-range and unsupported ones included
                std::vector<int32_t> sid((size_t)B);
                for (auto& v : sid) v = (int32_t)(rng() % (table.size() + 2)) - 1;
                Plan mixed;
                if (lower(model, B, sid.data(), 0, kMaxSlots, kMaxSlots, true, table, mixed, err, es)) ++lowered;
                else ++lower_refused;
                for (auto& v : sid) v = (int32_t)(rng() % table.size());
                if (lower(model, B, sid.data(), 0, 3, 3, true, table, mixed, err, es)) ++lowered;
                else ++lower_refused;
            }
        }
    }
    // random node arrays straight into the compiler
    long random_ok = 0, random_bad = 0;
    for (int t = 0; t < 20000; ++t) {
        const int n = 1 + (int)(rng() % 70);
        std::vector<kgq_node> g((size_t)n);
        for (int i = 0; i < n; ++i) {
            g[i].op = (int32_t)(rng() % 7) - 1;
            g[i].slot = (int32_t)(rng() % 12) - 2;
            for (int j = 0; j < 4; ++j) g[i].in[j] = (rng() % 3) ? (int32_t)(rng() % (n + 3)) - 2 : -1;
        }
        Program P;
        std::string err;
        int st = 0;
        if (compile_graph((int)(rng() % 5), g.data(), n, "r", P, err, st)) ++random_ok;
        else ++random_bad;
    }
    std::printf("parsed %ld rejected %ld compiled %ld lowered %ld refused %ld random accepted %ld rejected %ld\n",
                parsed, rejected, compiled, lowered, lower_refused, random_ok, random_bad);
    return 0;
}
