// Profiling driver: a plain C++ program that loads synthetic layers saved by
// `python3 -m paper_2609_04244_amd.profile_layer generate`, copies them to the GPU and
// launches the fused operator through the C ABI only (no other runtime in the process),
// followed by the reference copy/read kernels.  Used under rocprofv3 for kernel traces
// and hardware counters.
//
//   monomoe_profile DIR T_LIST ITERS COPY_MIB
//     DIR       directory with meta.txt and l<l>_<field>.bin
//     T_LIST    comma-separated token counts, e.g. 1,8
//     ITERS     launches per token count (layers rotate)
//     COPY_MIB  size of the reference copy/read kernels (0 = skip)
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/monomoe.h"

namespace {

bool read_file(const std::string& path, std::vector<char>& buf) {
    FILE* f = fopen(path.c_str(), "rb");
    if (!f) return false;
    fseek(f, 0, SEEK_END);
    const long n = ftell(f);
    fseek(f, 0, SEEK_SET);
    buf.resize((size_t)n);
    const size_t got = n > 0 ? fread(buf.data(), 1, (size_t)n, f) : 0;
    fclose(f);
    return got == (size_t)n;
}

void* to_device(const std::vector<char>& h) {
    void* d = nullptr;
    if (hipMalloc(&d, h.size() ? h.size() : 16) != hipSuccess) return nullptr;
    if (!h.empty() && hipMemcpy(d, h.data(), h.size(), hipMemcpyHostToDevice) != hipSuccess) return nullptr;
    return d;
}

int fail(const char* what) {
    fprintf(stderr, "monomoe_profile: %s\n", what);
    return 1;
}

}  // namespace

int main(int argc, char** argv) {
    if (argc != 5) return fail("usage: monomoe_profile DIR T_LIST ITERS COPY_MIB");
    const std::string dir = argv[1];
    const int iters = atoi(argv[3]);
    const size_t copy_mib = (size_t)atoll(argv[4]);
    int H, E, I, k, renorm, layers, tmax, has_bias;
    {
        FILE* f = fopen((dir + "/meta.txt").c_str(), "r");
        if (!f) return fail("cannot open meta.txt");
        const int n = fscanf(f, "%d %d %d %d %d %d %d %d", &H, &E, &I, &k, &renorm, &layers, &tmax, &has_bias);
        fclose(f);
        if (n != 8) return fail("bad meta.txt");
    }
    const char* fields[7] = {"x", "router_w", "bias", "w13", "w13_scale", "w2", "w2_scale"};
    std::vector<std::vector<void*>> dev(layers, std::vector<void*>(7, nullptr));
    for (int l = 0; l < layers; ++l) {
        for (int f = 0; f < 7; ++f) {
            if (f == 2 && !has_bias) continue;
            std::vector<char> h;
            const std::string path = dir + "/l" + std::to_string(l) + "_" + fields[f] + ".bin";
            if (!read_file(path, h)) return fail(("cannot read " + path).c_str());
            dev[l][f] = to_device(h);
            if (!dev[l][f]) return fail("device copy failed");
        }
    }
    char* list = argv[2];
    for (char* tok = strtok(list, ","); tok; tok = strtok(nullptr, ",")) {
        const int T = atoi(tok);
        if (T < 1 || T > tmax) return fail("token count out of range");
        monomoe_shape_t shape = {T, H, E, I};
        monomoe_plan_t plan = nullptr;
        int rc = monomoe_plan(&shape, k, renorm, &plan);
        if (rc != MONOMOE_OK) return fail(monomoe_status_string(rc));
        void* out = nullptr;
        if (hipMalloc(&out, (size_t)T * H * 2) != hipSuccess) return fail("hipMalloc out");
        for (int i = 0; i < iters; ++i) {
            const std::vector<void*>& L = dev[i % layers];
            monomoe_plan_set_router_bias(plan, static_cast<const float*>(L[2]));
            rc = monomoe_forward(plan, L[0], L[1], L[3], static_cast<const float*>(L[4]), L[5],
                                 static_cast<const float*>(L[6]), out, nullptr);
            if (rc != MONOMOE_OK) return fail(monomoe_status_string(rc));
        }
        if (hipDeviceSynchronize() != hipSuccess) return fail("synchronize");
        rc = monomoe_plan_status(plan);
        printf("T=%d: %d launches, device status %s\n", T, iters, monomoe_status_string(rc));
        fflush(stdout);
        monomoe_plan_destroy(plan);
        (void)hipFree(out);
        if (rc != MONOMOE_OK) return 1;
    }
    if (copy_mib) {
        const size_t n = copy_mib << 20;
        void *src = nullptr, *dst = nullptr, *sink = nullptr;
        if (hipMalloc(&src, n) != hipSuccess || hipMalloc(&dst, n) != hipSuccess || hipMalloc(&sink, 16) != hipSuccess)
            return fail("hipMalloc reference buffers");
        for (int r = 0; r < 3; ++r) monomoe_stream_copy(dst, src, n, nullptr);
        for (int r = 0; r < 3; ++r) monomoe_stream_read(src, n, sink, nullptr);
        if (hipDeviceSynchronize() != hipSuccess) return fail("synchronize");
        printf("reference copy and read kernels: %zu MiB each, 3 launches\n", copy_mib);
    }
    return 0;
}
