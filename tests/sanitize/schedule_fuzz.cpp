// Host-only driver for the sanitizer run of the integer schedules: reads
// test cases (one per line), runs the library's schedule builders on them
// and prints the status and the schedule.  Built with AddressSanitizer and
// UndefinedBehaviorSanitizer next to paper_1812_01329_amd/csrc/schedule.cpp
// alone (no device code), and compared with the oracle's schedules by
// tests/test_schedule_sanitized.py.
//
// Input lines (space-separated integers):
//   S B T has_lengths lengths[B]
//   T V N K left[N] right[N] word[N] root[K]
//   N V N K E offsets[N + 1] children[E] word[N] root[K]
// Output: one line per case, the status, then for a valid input the arrays
// separated by " |".
#include <cstdio>
#include <fstream>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "../../paper_1812_01329_amd/csrc/runtime.hpp"

namespace {

std::vector<int32_t> take(std::istringstream& in, long n) {
    std::vector<int32_t> v;
    for (long i = 0; i < n; ++i) {
        long x = 0;
        in >> x;
        v.push_back(int32_t(x));
    }
    return v;
}

void put(std::ostringstream& out, const int32_t* p, long n) {
    out << " |";
    for (long i = 0; i < n; ++i) out << ' ' << p[i];
}

}  // namespace

int main(int argc, char** argv) {
    if (argc != 3) {
        std::fprintf(stderr, "usage: %s cases.txt results.txt\n", argv[0]);
        return 2;
    }
    std::ifstream in(argv[1]);
    std::ofstream res(argv[2]);
    std::string line;
    long cases = 0;
    while (std::getline(in, line)) {
        std::istringstream is(line);
        std::string kind;
        is >> kind;
        std::ostringstream out;
        if (kind == "S") {
            long B = 0, T = 0, has = 0;
            is >> B >> T >> has;
            std::vector<int32_t> len = has ? take(is, B) : std::vector<int32_t>();
            janus::SeqSchedule s;
            const janus_status st = janus::build_seq_schedule(int32_t(B), int32_t(T), has ? len.data() : nullptr, s);
            out << int(st);
            if (st == JANUS_OK) {
                put(out, s.perm.data(), B);
                put(out, s.active.data(), s.t_eff);
                put(out, s.offsets.data(), s.t_eff + 1);
                out << " | " << s.t_eff;
            }
        } else if (kind == "T") {
            long V = 0, N = 0, K = 0;
            is >> V >> N >> K;
            std::vector<int32_t> left = take(is, N), right = take(is, N), word = take(is, N), root = take(is, K);
            janus_tree_batch t{int32_t(K), int32_t(N), left.data(), right.data(), word.data(), root.data()};
            janus::TreeSchedule s;
            const janus_status st = janus::build_tree_schedule(&t, int32_t(V), s);
            out << int(st);
            if (st == JANUS_OK) {
                put(out, s.level.data(), N);
                put(out, s.level_offsets.data(), s.num_levels + 1);
                put(out, s.level_nodes.data(), N);
            }
        } else if (kind == "N") {
            long V = 0, N = 0, K = 0, E = 0;
            is >> V >> N >> K >> E;
            std::vector<int32_t> off = take(is, N + 1), ch = take(is, E), word = take(is, N), root = take(is, K);
            janus_nary_tree_batch t{};
            t.num_trees = int32_t(K);
            t.num_nodes = int32_t(N);
            t.child_offsets = off.data();
            t.children = E > 0 ? ch.data() : nullptr;
            t.word = word.data();
            t.root = root.data();
            janus::NarySchedule s;
            const janus_status st = janus::build_nary_schedule(&t, int32_t(V), s);
            out << int(st);
            if (st == JANUS_OK) {
                put(out, s.level_offsets.data(), long(s.level_offsets.size()));
                put(out, s.pword.data(), N);
                put(out, s.pcoff.data(), N + 1);
                put(out, s.pkids.data(), E);
                put(out, s.rootk.data(), N);
                put(out, s.rootpos.data(), K);
            }
        } else {
            continue;
        }
        res << out.str() << '\n';
        ++cases;
    }
    std::printf("%ld cases\n", cases);
    return 0;
}
