// graph_host_check.cpp -- host-only harness of the graph index builder
// (csrc/graph.cpp + csrc/status.cpp), built with g++ under AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_graph_sanitize.py.
//
// No HIP runtime is linked: the few runtime calls the builder makes on its
// device path are defined below to report "no device", and every graph here
// is created with RGNN_GRAPH_HOST_ONLY, so none of them is reached.
//
// Global operator new is replaced by a counting version that can be armed to
// fail exactly one allocation; the leak checker at exit then shows whether
// the builder released everything on that error path.
//
// Modes:
//   index <in> <out>   build the graph described by <in> (see read_graph) and
//                      write its info and every exported index array to <out>
//   errors             invalid inputs -> the documented status codes
//   nomem <in>         fail the k-th allocation of a graph creation, for every
//                      k until a creation runs without failure
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include <hip/hip_runtime_api.h>

#include "rgnn.h"

// ---------------------------------------------------------------- no device
hipError_t hipMalloc(void **p, size_t) { if (p) *p = nullptr; return hipErrorNoDevice; }
hipError_t hipFree(void *) { return hipErrorNoDevice; }
hipError_t hipMemcpy(void *, const void *, size_t, hipMemcpyKind) { return hipErrorNoDevice; }
hipError_t hipMemcpyAsync(void *, const void *, size_t, hipMemcpyKind, hipStream_t) { return hipErrorNoDevice; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipErrorNoDevice; }
hipError_t hipGetDevice(int *d) { if (d) *d = -1; return hipErrorNoDevice; }
hipError_t hipSetDevice(int) { return hipErrorNoDevice; }
const char *hipGetErrorString(hipError_t) { return "no device in the host-only harness"; }

// ---------------------------------------------------------------- allocation failure injection
static long g_alloc_count = 0;     // allocations since arming
static long g_fail_at = 0;         // fail the allocation with this count (0: never)
static bool g_fired = false;

static void *counted_alloc(size_t n, bool nothrow)
{
    if (g_fail_at > 0 && ++g_alloc_count == g_fail_at) {
        g_fired = true;
        if (nothrow) return nullptr;
        throw std::bad_alloc();
    }
    void *p = std::malloc(n ? n : 1);
    if (!p && !nothrow) throw std::bad_alloc();
    return p;
}

void *operator new(size_t n) { return counted_alloc(n, false); }
void *operator new[](size_t n) { return counted_alloc(n, false); }
void *operator new(size_t n, const std::nothrow_t &) noexcept { return counted_alloc(n, true); }
void *operator new[](size_t n, const std::nothrow_t &) noexcept { return counted_alloc(n, true); }
void operator delete(void *p) noexcept { std::free(p); }
void operator delete[](void *p) noexcept { std::free(p); }
void operator delete(void *p, size_t) noexcept { std::free(p); }
void operator delete[](void *p, size_t) noexcept { std::free(p); }
void operator delete(void *p, const std::nothrow_t &) noexcept { std::free(p); }
void operator delete[](void *p, const std::nothrow_t &) noexcept { std::free(p); }

// ---------------------------------------------------------------- input
struct GraphIn {
    int64_t N = 0, E = 0;
    int32_t T = 1, R = 1, csr = 0, flags = 0;
    std::vector<int32_t> src, dst, rel, ntype;
    std::vector<int64_t> rowptr;
};

// <in>: int64 N, int64 E, int32 T, int32 R, int32 csr, int32 flags, then
//   COO: src, dst, rel [E] int32, ntype [N] int32
//   CSR: rowptr [N+1] int64, col_src, rel [E] int32, ntype [N] int32
static bool read_graph(const char *path, GraphIn &g)
{
    FILE *f = std::fopen(path, "rb");
    if (!f) return false;
    bool ok = std::fread(&g.N, 8, 1, f) == 1 && std::fread(&g.E, 8, 1, f) == 1 &&
              std::fread(&g.T, 4, 1, f) == 1 && std::fread(&g.R, 4, 1, f) == 1 &&
              std::fread(&g.csr, 4, 1, f) == 1 && std::fread(&g.flags, 4, 1, f) == 1;
    if (ok && g.csr) {
        g.rowptr.resize((size_t)g.N + 1);
        ok = std::fread(g.rowptr.data(), 8, g.rowptr.size(), f) == g.rowptr.size();
    }
    g.src.resize((size_t)g.E);
    g.rel.resize((size_t)g.E);
    g.ntype.resize((size_t)g.N);
    ok = ok && std::fread(g.src.data(), 4, g.src.size(), f) == g.src.size();
    if (ok && !g.csr) {
        g.dst.resize((size_t)g.E);
        ok = std::fread(g.dst.data(), 4, g.dst.size(), f) == g.dst.size();
    }
    ok = ok && std::fread(g.rel.data(), 4, g.rel.size(), f) == g.rel.size() &&
         std::fread(g.ntype.data(), 4, g.ntype.size(), f) == g.ntype.size();
    std::fclose(f);
    return ok;
}

static rgnn_status create(const GraphIn &g, rgnn_graph_t **out)
{
    const int32_t flags = g.flags | RGNN_GRAPH_HOST_ONLY;
    if (g.csr)
        return rgnn_graph_create_csr(g.N, g.T, g.R, g.rowptr.data(), g.src.data(), g.rel.data(),
                                     g.ntype.data(), flags, nullptr, out);
    return rgnn_graph_create_coo(g.N, g.T, g.R, g.E, g.src.data(), g.dst.data(), g.rel.data(),
                                 g.ntype.data(), flags, nullptr, out);
}

// ---------------------------------------------------------------- modes
static int mode_index(const char *in, const char *outp)
{
    GraphIn g;
    if (!read_graph(in, g)) { std::fprintf(stderr, "cannot read %s\n", in); return 2; }
    rgnn_graph_t *G = nullptr;
    rgnn_status st = create(g, &G);
    if (st != RGNN_OK) { std::fprintf(stderr, "create: %d %s\n", (int)st, rgnn_last_error()); return 3; }
    rgnn_graph_info_t inf;
    if (rgnn_graph_info(G, &inf) != RGNN_OK) return 4;
    FILE *f = std::fopen(outp, "wb");
    if (!f) return 2;
    const int64_t head[4] = {inf.num_src_pairs, inf.num_dst_segments, inf.max_in_degree, inf.num_empty_dst};
    std::fwrite(head, 8, 4, f);
    const int64_t N = inf.num_nodes, E = inf.num_edges, U = inf.num_src_pairs, S = inf.num_dst_segments;
    const int64_t sizes[14] = {N + 1, E, E, E, S + 1, S, N + 1, U, inf.num_rels + 1, E, N,
                               inf.num_ntypes + 1, N + 1, E};
    int rc = 0;
    for (int k = 0; k < 14 && !rc; ++k) {
        std::vector<int32_t> buf((size_t)sizes[k] + 1, -7);
        st = rgnn_graph_export(G, k, buf.data(), (size_t)sizes[k] * 4);
        if (st != RGNN_OK) { std::fprintf(stderr, "export %d: %s\n", k, rgnn_last_error()); rc = 5; }
        if (buf[(size_t)sizes[k]] != -7) { std::fprintf(stderr, "export %d wrote past its size\n", k); rc = 6; }
        std::fwrite(&sizes[k], 8, 1, f);
        std::fwrite(buf.data(), 4, (size_t)sizes[k], f);
    }
    std::fclose(f);
    if (rgnn_graph_destroy(G) != RGNN_OK) rc = 7;
    return rc;
}

static int expect(const char *what, rgnn_status got, rgnn_status want, rgnn_graph_t **G)
{
    const bool ok = got == want && (want == RGNN_OK || std::strlen(rgnn_last_error()) > 0);
    std::printf("%s %s: %d (want %d) %s\n", ok ? "ok" : "FAIL", what, (int)got, (int)want,
                want == RGNN_OK ? "" : rgnn_last_error());
    if (G && *G) {   // read after the call that set it
        rgnn_graph_destroy(*G);
        *G = nullptr;
    }
    return ok ? 0 : 1;
}

static int mode_errors()
{
    const int32_t src[4] = {0, 1, 2, 1}, dst[4] = {1, 2, 0, 0}, rel[4] = {0, 1, 0, 1}, nt[3] = {0, 1, 0};
    const int H = RGNN_GRAPH_HOST_ONLY;
    int bad = 0;
    rgnn_graph_t *G = nullptr;
    bad += expect("valid", rgnn_graph_create_coo(3, 2, 2, 4, src, dst, rel, nt, H, nullptr, &G), RGNN_OK, &G);
    bad += expect("out NULL", rgnn_graph_create_coo(3, 2, 2, 4, src, dst, rel, nt, H, nullptr, nullptr), RGNN_EINVAL, nullptr);
    bad += expect("N < 0", rgnn_graph_create_coo(-1, 2, 2, 4, src, dst, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("E < 0", rgnn_graph_create_coo(3, 2, 2, -4, src, dst, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("E >= 2^31", rgnn_graph_create_coo(3, 2, 2, int64_t(1) << 31, src, dst, rel, nt, H, nullptr, &G), RGNN_ERANGE, &G);
    bad += expect("R = 0", rgnn_graph_create_coo(3, 2, 0, 4, src, dst, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("T = 0", rgnn_graph_create_coo(3, 0, 2, 4, src, dst, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("src NULL", rgnn_graph_create_coo(3, 2, 2, 4, nullptr, dst, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("unknown flag", rgnn_graph_create_coo(3, 2, 2, 4, src, dst, rel, nt, H | 64, nullptr, &G), RGNN_EINVAL, &G);
    const int32_t bsrc[4] = {0, 3, 2, 1}, bdst[4] = {1, 2, -1, 0}, brel[4] = {0, 1, 2, 1}, bnt[3] = {0, 2, 0};
    bad += expect("src out of range", rgnn_graph_create_coo(3, 2, 2, 4, bsrc, dst, rel, nt, H, nullptr, &G), RGNN_ERANGE, &G);
    bad += expect("dst out of range", rgnn_graph_create_coo(3, 2, 2, 4, src, bdst, rel, nt, H, nullptr, &G), RGNN_ERANGE, &G);
    bad += expect("rel out of range", rgnn_graph_create_coo(3, 2, 2, 4, src, dst, brel, nt, H, nullptr, &G), RGNN_ERANGE, &G);
    bad += expect("ntype out of range", rgnn_graph_create_coo(3, 2, 2, 4, src, dst, rel, bnt, H, nullptr, &G), RGNN_ERANGE, &G);
    bad += expect("no edges", rgnn_graph_create_coo(3, 2, 2, 0, nullptr, nullptr, nullptr, nullptr, H, nullptr, &G), RGNN_OK, &G);
    const int64_t rp_ok[4] = {0, 2, 3, 4}, rp_nonmono[4] = {0, 2, 1, 4}, rp_first[4] = {1, 2, 3, 4};
    bad += expect("csr valid", rgnn_graph_create_csr(3, 2, 2, rp_ok, src, rel, nt, H, nullptr, &G), RGNN_OK, &G);
    bad += expect("csr not monotone", rgnn_graph_create_csr(3, 2, 2, rp_nonmono, src, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("csr rowptr[0] != 0", rgnn_graph_create_csr(3, 2, 2, rp_first, src, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("csr rowptr NULL", rgnn_graph_create_csr(3, 2, 2, nullptr, src, rel, nt, H, nullptr, &G), RGNN_EINVAL, &G);
    bad += expect("csr out NULL", rgnn_graph_create_csr(3, 2, 2, rp_ok, src, rel, nt, H, nullptr, nullptr), RGNN_EINVAL, nullptr);
    // calls on a valid host-only graph
    rgnn_graph_create_coo(3, 2, 2, 4, src, dst, rel, nt, H, nullptr, &G);
    int32_t small[2];
    bad += expect("export too small", rgnn_graph_export(G, RGNN_IDX_IN_SRC, small, sizeof small), RGNN_EINVAL, nullptr);
    bad += expect("export unknown kind", rgnn_graph_export(G, 99, small, sizeof small), RGNN_EINVAL, nullptr);
    bad += expect("export NULL", rgnn_graph_export(G, RGNN_IDX_IN_SRC, nullptr, 64), RGNN_EINVAL, nullptr);
    bad += expect("info NULL", rgnn_graph_info(G, nullptr), RGNN_EINVAL, nullptr);
    bad += expect("info of NULL graph", rgnn_graph_info(nullptr, nullptr), RGNN_EINVAL, nullptr);
    bad += expect("destroy NULL", rgnn_graph_destroy(nullptr), RGNN_OK, nullptr);
    bad += expect("destroy", rgnn_graph_destroy(G), RGNN_OK, nullptr);
    G = nullptr;
    return bad ? 1 : 0;
}

static int mode_nomem(const char *in)
{
    GraphIn g;
    if (!read_graph(in, g)) { std::fprintf(stderr, "cannot read %s\n", in); return 2; }
    long k = 1, n_nomem = 0;
    for (;; ++k) {
        rgnn_graph_t *G = nullptr;
        g_alloc_count = 0;
        g_fired = false;
        g_fail_at = k;
        const rgnn_status st = create(g, &G);
        g_fail_at = 0;
        if (g_fired) {
            if (st != RGNN_ENOMEM || G != nullptr) {
                std::printf("FAIL allocation %ld failed: status %d, graph %p\n", k, (int)st, (void *)G);
                return 1;
            }
            ++n_nomem;
            continue;
        }
        if (st != RGNN_OK) { std::printf("FAIL status %d without a failed allocation\n", (int)st); return 1; }
        rgnn_graph_destroy(G);
        break;
    }
    std::printf("ok %ld allocations, each failure returned RGNN_ENOMEM\n", n_nomem);
    return n_nomem > 0 ? 0 : 1;
}

int main(int argc, char **argv)
{
    if (argc >= 4 && !std::strcmp(argv[1], "index")) return mode_index(argv[2], argv[3]);
    if (argc >= 2 && !std::strcmp(argv[1], "errors")) return mode_errors();
    if (argc >= 3 && !std::strcmp(argv[1], "nomem")) return mode_nomem(argv[2]);
    std::fprintf(stderr, "usage: %s index <in> <out> | errors | nomem <in>\n", argv[0]);
    return 2;
}
