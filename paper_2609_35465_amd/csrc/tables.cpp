// Host-side construction of the Tetra decoder tables (see tables.h).
//
// Conventions fixed here where the paper is silent:
//  * Golay code: cyclic [23,12] code with generator polynomial
//    1 + x^2 + x^4 + x^5 + x^6 + x^10 + x^11 (bits 0xC75), extended by an
//    overall parity bit at coordinate 23.
//  * Trio: octad 1 has the lexicographically smallest sorted support,
//    octad 2 the smallest one disjoint from it, octad 3 is the rest.
//    Section s, position t is the t-th smallest coordinate of octad s+1.
//  * Trellis numbering: s8 numbers the complementary pairs {P, P^0xFF} of
//    section-1 bytes by ascending min(P, P^0xFF); b1 = 0 picks the smaller
//    byte.  s16 numbers section-3 pairs the same way.  The 16 branches of
//    s8 are its continuations (P2, s16) in ascending order of P2.
//  * Rank table: the 2,048 cheapest rank vectors of each class, ordered by
//    (cost, packed 32-bit row) ascending; the middle list is the 2,048
//    cheapest overall under the same order, class 0 first.
//  * gain = {4.3f, 5.4f}.
#include "tables.h"

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <mutex>
#include <set>
#include <stdexcept>
#include <utility>

namespace tetra {
namespace {

constexpr uint32_t kGolayGen = 0xC75u;

int popcount32(uint32_t v) { return __builtin_popcount(v); }

std::vector<uint32_t> golay_codewords() {
    std::vector<uint32_t> out;
    out.reserve(4096);
    for (uint32_t msg = 0; msg < 4096; ++msg) {
        uint32_t c = 0;
        for (int i = 0; i < 12; ++i)
            if (msg >> i & 1u) c ^= kGolayGen << i;      // msg(x) * g(x)
        c |= static_cast<uint32_t>(popcount32(c) & 1) << 23;
        out.push_back(c);
    }
    return out;
}

using Octad = std::array<int, 8>;

Octad support_of(uint32_t c) {
    Octad o{};
    int n = 0;
    for (int i = 0; i < 24; ++i)
        if (c >> i & 1u) o[n++] = i;
    return o;
}

// sec[s][t]: original coordinate of section s, position t
std::array<std::array<int, 8>, 3> octad_trio(const std::vector<uint32_t>& code) {
    std::vector<std::pair<Octad, uint32_t>> octads;
    for (uint32_t c : code)
        if (popcount32(c) == 8) octads.push_back({support_of(c), c});
    std::sort(octads.begin(), octads.end());
    const uint32_t m1 = octads.front().second;
    uint32_t m2 = 0;
    for (auto& o : octads)
        if ((o.second & m1) == 0) { m2 = o.second; break; }
    const uint32_t m3 = ~(m1 | m2) & 0xFFFFFFu;
    std::array<std::array<int, 8>, 3> sec{};
    const uint32_t masks[3] = {m1, m2, m3};
    for (int s = 0; s < 3; ++s) {
        if (popcount32(masks[s]) != 8) throw std::runtime_error("trio: not an octad");
        sec[s] = support_of(masks[s]);
    }
    return sec;
}

uint8_t pair_rep(uint8_t b) { return std::min<uint8_t>(b, static_cast<uint8_t>(b ^ 0xFFu)); }

struct RankCand { uint32_t cost, packed; };

bool operator<(const RankCand& a, const RankCand& b) {
    return a.cost != b.cost ? a.cost < b.cost : a.packed < b.packed;
}

// Visits every rank vector in {0..7}^8 as (packed row, cost, class).
template <class F> void for_each_rank_vector(F&& f) {
    for (uint32_t idx = 0; idx < (1u << 24); ++idx) {
        uint32_t packed = 0, cost = 0, cls = 0;
        for (int j = 0; j < 8; ++j) {
            const uint32_t d = idx >> (3 * j) & 7u;
            packed |= d << (4 * j);
            cost += (2 * d + 1) * (2 * d + 1);
            cls ^= (d == 1 || d == 2 || d == 5 || d == 6);
        }
        f(packed, cost, cls);
    }
}

// The n cheapest vectors accepted by `want`, in (cost, packed) order.
template <class Pred> std::vector<RankCand> cheapest(int n, Pred want) {
    // pass 1: cost histogram of the accepted vectors, to find the cut cost
    std::vector<uint32_t> hist(8 * 225 + 1, 0);
    for_each_rank_vector([&](uint32_t, uint32_t cost, uint32_t cls) {
        if (want(cls)) ++hist[cost];
    });
    uint32_t cut = 0, acc = 0;
    while (acc < static_cast<uint32_t>(n)) acc += hist[cut++];
    // pass 2: gather everything at or below the cut, sort, keep n
    std::vector<RankCand> v;
    for_each_rank_vector([&](uint32_t packed, uint32_t cost, uint32_t cls) {
        if (want(cls) && cost < cut) v.push_back({cost, packed});
    });
    std::sort(v.begin(), v.end());
    v.resize(n);
    return v;
}

void build(HostTables& T) {
    std::memset(&T, 0, sizeof(T));
    const auto code = golay_codewords();
    const auto sec = octad_trio(code);

    auto section_byte = [&](uint32_t c, int s) {
        uint32_t b = 0;
        for (int t = 0; t < 8; ++t) b |= (c >> sec[s][t] & 1u) << t;
        return static_cast<uint8_t>(b);
    };

    // trellis states
    std::set<uint8_t> reps1, reps3;
    for (uint32_t c : code) {
        reps1.insert(pair_rep(section_byte(c, 0)));
        reps3.insert(pair_rep(section_byte(c, 2)));
    }
    if (reps1.size() != 64 || reps3.size() != 64) throw std::runtime_error("trellis: states");
    int s8_of[256], s16_of[256];
    std::fill(s8_of, s8_of + 256, -1);
    std::fill(s16_of, s16_of + 256, -1);
    int k = 0;
    for (uint8_t r : reps1) { s8_of[r] = s8_of[r ^ 0xFF] = k; T.prefixes[2 * k] = r; T.prefixes[2 * k + 1] = r ^ 0xFF; ++k; }
    k = 0;
    for (uint8_t r : reps3) { s16_of[r] = s16_of[r ^ 0xFF] = k; T.suffixes[2 * k] = r; T.suffixes[2 * k + 1] = r ^ 0xFF; ++k; }

    std::array<std::set<std::pair<int, int>>, 64> cont;
    for (uint32_t c : code)
        cont[s8_of[section_byte(c, 0)]].insert({section_byte(c, 1), s16_of[section_byte(c, 2)]});
    for (int s8 = 0; s8 < 64; ++s8) {
        if (cont[s8].size() != 16) throw std::runtime_error("trellis: branches");
        int b2 = 0;
        for (auto& e : cont[s8])
            T.branches[16 * s8 + b2++] = static_cast<uint16_t>(e.first | e.second << 8);
    }

    // every path, and a check that the paths are exactly the code
    std::set<uint32_t> codeset(code.begin(), code.end()), seen;
    for (int s8 = 0; s8 < 64; ++s8)
        for (int b1 = 0; b1 < 2; ++b1)
            for (int b2 = 0; b2 < 16; ++b2)
                for (int b3 = 0; b3 < 2; ++b3) {
                    const uint32_t p1 = T.prefixes[2 * s8 + b1];
                    const uint32_t br = T.branches[16 * s8 + b2];
                    const uint32_t p2 = br & 0xFFu, s16 = br >> 8;
                    const uint32_t p3 = T.suffixes[2 * s16 + b3];
                    T.path_bytes[s8 | b1 << 6 | b2 << 7 | b3 << 11] = p1 | p2 << 8 | p3 << 16;
                    uint32_t c = 0;
                    const uint32_t bytes[3] = {p1, p2, p3};
                    for (int s = 0; s < 3; ++s)
                        for (int t = 0; t < 8; ++t) c |= (bytes[s] >> t & 1u) << sec[s][t];
                    if (!codeset.count(c)) throw std::runtime_error("trellis: path not a codeword");
                    seen.insert(c);
                }
    if (seen.size() != 4096) throw std::runtime_error("trellis: paths not a bijection");

    // rank table and middle list
    const auto h0 = cheapest(kHalfRows, [](uint32_t cls) { return cls == 0; });
    const auto h1 = cheapest(kHalfRows, [](uint32_t cls) { return cls == 1; });
    for (int i = 0; i < kHalfRows; ++i) { T.rows[i] = h0[i].packed; T.rows[kHalfRows + i] = h1[i].packed; }
    const auto all = cheapest(kHalfRows, [](uint32_t) { return true; });
    std::vector<uint32_t> mid;
    for (int pass = 0; pass < 2; ++pass)
        for (auto& r : all) {
            uint32_t cls = 0;
            for (int j = 0; j < 8; ++j) {
                const uint32_t d = r.packed >> (4 * j) & 15u;
                cls ^= (d == 1 || d == 2 || d == 5 || d == 6);
            }
            if (static_cast<int>(cls) == pass) mid.push_back(r.packed);
            if (pass == 0 && cls == 0) ++T.n_mid_class0;
        }
    if (T.n_mid_class0 != kMidClass0) throw std::runtime_error("rank table: middle split");
    for (int i = 0; i < kHalfRows; ++i) {
        const int phys = i < kMidClass0 ? i : kHalfRows + (i - kMidClass0);
        if (T.rows[phys] != mid[i]) throw std::runtime_error("rank table: middle list is not a prefix");
    }

    T.invnorm[0] = 0.0f;
    for (int m = 1; m < 32; ++m) T.invnorm[m] = static_cast<float>(1.0 / std::sqrt(16.0 * m));
    T.gain[0] = 4.3f;
    T.gain[1] = 5.4f;
}

}  // namespace

const HostTables& host_tables() {
    static HostTables T;
    static std::once_flag once;
    std::call_once(once, [] { build(T); });
    return T;
}

std::vector<uint8_t> canonical_blob() {
    const HostTables& T = host_tables();
    std::vector<uint8_t> out;
    auto put = [&](const void* p, size_t n) {
        const uint8_t* b = static_cast<const uint8_t*>(p);
        out.insert(out.end(), b, b + n);
    };
    put(T.rows, sizeof(T.rows));
    put(T.branches, sizeof(T.branches));
    put(T.prefixes, sizeof(T.prefixes));
    put(T.suffixes, sizeof(T.suffixes));
    put(T.invnorm, sizeof(T.invnorm));
    put(T.gain, sizeof(T.gain));
    return out;   // x86-64 host: already little-endian
}

}  // namespace tetra
