// Build-time generator of the device decoder tables: runs the host table
// construction (tables.cpp), lays the tables out as the kernels read them
// (table_layout.h) and prints them as the initialisers of the library's
// constant device tables.  Host code only.
//
// Usage: gen_tables > tables_data.inc
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <vector>

#include "table_layout.h"

namespace {

void words(const uint32_t* w, size_t n) {
    for (size_t i = 0; i < n; ++i) std::printf("%s0x%08xu%s", i % 8 ? " " : " \\\n    ", w[i], i + 1 < n ? "," : "");
}

void floats(const float* f, size_t n) {
    for (size_t i = 0; i < n; ++i) std::printf("%s%af%s", i % 4 ? " " : " \\\n    ", static_cast<double>(f[i]), i + 1 < n ? "," : "");
}

}  // namespace

int main() {
    const tetra::HostTables& T = tetra::host_tables();
    std::vector<uint8_t> buf(sizeof(tetra_dev::CanonicalTables) + sizeof(tetra_dev::PackedTables));
    auto* c = reinterpret_cast<tetra_dev::CanonicalTables*>(buf.data());
    auto* p = reinterpret_cast<tetra_dev::PackedTables*>(buf.data() + sizeof(tetra_dev::CanonicalTables));
    tetra_dev::build_canonical(T, c);
    tetra_dev::build_packed(T, p);
    std::printf("// Generated at build time by gen_tables.cpp from the host table construction; do not edit.\n");
    std::printf("#define TETRA_CANONICAL_TABLES_INIT { {");
    words(c->path_bytes, 4096);
    std::printf("}, {");
    words(c->rows, 4096);
    std::printf("}, {");
    floats(c->invnorm, 32);
    std::printf("}, {");
    floats(c->gain, 2);
    std::printf("}, {0u, 0u} }\n");
    std::printf("#define TETRA_PACKED_TABLES_INIT { {");
    words(p->path_e, 4096);
    std::printf("}, {");
    for (int i = 0; i < 4096; ++i)
        std::printf("%s{0x%08xu, 0x%08xu}%s", i % 4 ? " " : " \\\n    ", p->rows_f8[i][0], p->rows_f8[i][1],
                    i + 1 < 4096 ? "," : "");
    std::printf("}, {");
    floats(p->scale, sizeof(p->scale) / sizeof(float));
    std::printf("}, {");
    for (int i = 0; i < 4096; ++i) std::printf("%s%u%s", i % 16 ? " " : " \\\n    ", p->cost[i], i + 1 < 4096 ? "," : "");
    std::printf("} }\n");
    return 0;
}
