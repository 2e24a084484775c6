// Host-side exercise of the library under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_host_sanitizers.py with
// the sanitizers on the host code only, and run with no GPU visible):
// transfer-plan validation (valid plans reach the device upload and stop
// there; invalid ones are rejected) and the storage path's host writer,
// commit, chain and reader, including a corrupted chunk.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <string>
#include <vector>
#include <algorithm>
#include <sys/stat.h>
#include "dte.h"
#include "dte_store.h"

static int fails = 0;
#define CHECK(c) do { if (!(c)) { std::printf("FAIL %s:%d %s\n", __FILE__, __LINE__, #c); ++fails; } } while (0)

static dte_op op2(int seg, int rank, int64_t base, int64_t r0, int64_t nr, int64_t nc) {
    dte_op o; std::memset(&o, 0, sizeof o);
    o.segment = seg; o.rank = rank; o.dst_base = base;
    o.src_origin[0] = r0; o.extent[0] = nr; o.extent[1] = nc;
    o.dst_shape[0] = nr; o.dst_shape[1] = nc;
    return o;
}

int main(int argc, char** argv) {
    // plans
    dte_segment s[2]; std::memset(s, 0, sizeof s);
    s[0].flat_begin = 0; s[0].ndim = 2; s[0].shape[0] = 100; s[0].shape[1] = 30;
    s[1].flat_begin = 3000; s[1].ndim = 1; s[1].shape[0] = 77;
    std::vector<dte_op> ops = {op2(0, 0, 0, 0, 50, 30), op2(0, 1, 0, 50, 50, 30)};
    dte_op o; std::memset(&o, 0, sizeof o); o.segment = 1; o.rank = 0; o.dst_base = 1500; o.extent[0] = 77; o.dst_shape[0] = 77; ops.push_back(o);
    o.rank = 1; ops.push_back(o);
    int64_t numel[2] = {1577, 1577};
    dte_plan* p = nullptr;
    dte_status st = dte_plan_create(s, 2, ops.data(), (int)ops.size(), 2, numel, &p);
    std::printf("valid plan: %s\n", dte_status_string(st));
    CHECK(st == DTE_OK || st == DTE_ERR_HIP);
    if (p) dte_plan_destroy(p);
    ops[1].src_origin[0] = 40;   // overlaps rank 0? different rank: fine; but leaves rows uncovered? no: 40..90 -> rows 90..99 uncovered
    st = dte_plan_create(s, 2, ops.data(), (int)ops.size(), 2, numel, &p);
    CHECK(st == DTE_ERR_PLAN);
    ops[1].src_origin[0] = 50; ops[1].rank = 0;  // same rank twice in one view: overlapping destinations
    st = dte_plan_create(s, 2, ops.data(), (int)ops.size(), 2, numel, &p);
    CHECK(st == DTE_ERR_PLAN);
    // 4-D segment split in every dimension
    dte_segment s4; std::memset(&s4, 0, sizeof s4); s4.ndim = 4; s4.shape[0] = 5; s4.shape[1] = 6; s4.shape[2] = 7; s4.shape[3] = 8;
    std::vector<dte_op> o4;
    int64_t n4[16];
    for (int r = 0; r < 16; ++r) {
        dte_op q; std::memset(&q, 0, sizeof q); q.segment = 0; q.rank = r;
        const int64_t cut[4] = {(r & 1) ? 2 : 0, (r & 2) ? 3 : 0, (r & 4) ? 4 : 0, (r & 8) ? 5 : 0};
        for (int d = 0; d < 4; ++d) {
            const int64_t lo = cut[d], hi = cut[d] ? s4.shape[d] : (d == 0 ? 2 : d == 1 ? 3 : d == 2 ? 4 : 5);
            q.src_origin[d] = lo; q.extent[d] = hi - lo; q.dst_shape[d] = hi - lo;
        }
        int64_t v = 1; for (int d = 0; d < 4; ++d) v *= q.extent[d];
        n4[r] = v; o4.push_back(q);
    }
    st = dte_plan_create(&s4, 1, o4.data(), 16, 16, n4, &p);
    std::printf("4-D plan: %s\n", dte_status_string(st));
    CHECK(st == DTE_OK || st == DTE_ERR_HIP);
    if (p) dte_plan_destroy(p);

    // storage
    if (argc < 2) return 2;
    const std::string dir = argv[1];
    ::mkdir(dir.c_str(), 0755);
    dte_store_segment ss[3] = {{"a.weight", 0, 100000}, {"b.weight", 100000, 5000}, {"c", 105000, 70000}};
    std::mt19937_64 rng(7);
    for (int codec = 0; codec < 2; ++codec) {
        for (int tr = 0; tr < 2; ++tr) {
            const int64_t version = 1 + codec * 2 + tr;
            std::vector<int64_t> all;
            for (int64_t i = 0; i < 175000; ++i) if (rng() % 7 == 0) all.push_back(i);
            std::vector<int64_t> w0, w1; std::vector<uint16_t> v0, v1;
            for (int64_t x : all) { if (x < 100000) { w0.push_back(x); v0.push_back((uint16_t)(x * 31)); } else { w1.push_back(x); v1.push_back((uint16_t)(x * 31)); } }
            dte_store_options opt{codec, 3, 4, tr, 1000};
            dte_store_stats stats;
            st = dte_store_write_part_host(dir.c_str(), version, 0, ss, 3, w0.data(), v0.data(), (int64_t)w0.size(), &opt, &stats);
            if (st == DTE_ERR_UNSUPPORTED) { std::printf("zstd unavailable\n"); continue; }
            CHECK(st == DTE_OK);
            st = dte_store_write_part_host(dir.c_str(), version, 1, ss, 3, w1.data(), v1.data(), (int64_t)w1.size(), &opt, &stats);
            CHECK(st == DTE_OK);
            int32_t committed = 0;
            st = dte_store_commit(dir.c_str(), version, version - 1, 2, &committed);
            CHECK(st == DTE_OK && committed == 1);
            std::vector<int64_t> ri(all.size() + 10); std::vector<uint16_t> rv(all.size() + 10);
            int64_t cnt = 0;
            st = dte_store_read_host(dir.c_str(), version, version - 1, ri.data(), rv.data(), (int64_t)ri.size(), &cnt, 3, &stats);
            CHECK(st == DTE_OK && cnt == (int64_t)all.size());
            bool same = true;
            for (size_t i = 0; i < all.size(); ++i) same = same && ri[i] == all[i] && rv[i] == (uint16_t)(all[i] * 31);
            CHECK(same);
            // too small an output
            st = dte_store_read_host(dir.c_str(), version, version - 1, ri.data(), rv.data(), 5, &cnt, 2, &stats);
            CHECK(st == DTE_OK && cnt == (int64_t)all.size());
            std::printf("codec %d transform %d: %zu entries ok\n", codec, tr, all.size());
        }
    }
    int64_t latest = 0; st = dte_store_latest(dir.c_str(), &latest);
    CHECK(st == DTE_OK && latest >= 2);
    int64_t chain[8]; int32_t n = 0;
    st = dte_store_chain(dir.c_str(), 0, latest, chain, 8, &n);
    CHECK(st == DTE_OK && n == latest);
    st = dte_store_chain(dir.c_str(), 0, latest, chain, 1, &n);
    CHECK(st == DTE_ERR_ARG);
    // corrupt one chunk of version 1
    {
        std::string f = dir + "/v1/chunk-0-0.dte";
        FILE* fp = std::fopen(f.c_str(), "r+b");
        CHECK(fp != nullptr);
        if (fp) { std::fseek(fp, 45, SEEK_SET); int c = std::fgetc(fp); std::fseek(fp, 45, SEEK_SET); std::fputc(c ^ 0x55, fp); std::fclose(fp); }
        std::vector<int64_t> ri(200000); std::vector<uint16_t> rv(200000); int64_t cnt = 0; dte_store_stats stats;
        st = dte_store_read_host(dir.c_str(), 1, 0, ri.data(), rv.data(), 200000, &cnt, 2, &stats);
        CHECK(st == DTE_ERR_CORRUPT);
    }
    // empty parts publish nothing
    {
        dte_store_options opt{0, 3, 2, 1, 1000}; dte_store_stats stats; int32_t committed = 7;
        CHECK(dte_store_write_part_host(dir.c_str(), 50, 0, ss, 3, nullptr, nullptr, 0, &opt, &stats) == DTE_OK);
        CHECK(dte_store_commit(dir.c_str(), 50, 4, 1, &committed) == DTE_OK && committed == 0);
    }
    // unsorted input is rejected
    {
        int64_t bad[3] = {5, 3, 9}; uint16_t bv[3] = {1, 2, 3};
        dte_store_options opt{0, 3, 2, 1, 1000}; dte_store_stats stats;
        CHECK(dte_store_write_part_host(dir.c_str(), 60, 0, ss, 3, bad, bv, 3, &opt, &stats) == DTE_ERR_ARG);
    }
    std::printf("%s (%d failures)\n", fails ? "FAILED" : "ok", fails);
    return fails ? 1 : 0;
}
