// Drives the HIP library's host-only entry points and argument checks (no GPU
// needed); built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitizers.py.
#include <cstdio>
#include <cstdint>
#include <cmath>
#include <vector>
#include "lazytrain.h"
int main() {
    int bad = 0;
    // host-only entry points
    std::vector<int64_t> numels = {5, 100, 7, 300001, 2048, 65536};
    std::vector<uint8_t> is8(numels.size());
    int64_t chosen = 0;
    if (lt_select_8bit_slice(numels.data(), (int)numels.size(), 0.3, is8.data(), &chosen) != LT_OK) ++bad;
    if (lt_select_8bit_slice(numels.data(), (int)numels.size(), 1.5, is8.data(), &chosen) == LT_OK) ++bad;
    if (lt_grad_sqnorm_workspace_bytes(numels.data(), (int)numels.size()) == 0) ++bad;
    if (lt_step_workspace_bytes(-1) != 0 || lt_step_workspace_bytes(0) == 0 ||
        lt_step_workspace_bytes(7) == 0) ++bad;
    if (lt_grad_chunk_count(numels.data(), (int)numels.size()) != 1 + 1 + 1 + 37 + 1 + 8) ++bad;
    int first[3] = {0, 3, 6};
    for (int bf = 0; bf < 2; ++bf)
        for (int kg = 0; kg < 2; ++kg)
            if (lt_streamed_workspace_bytes(numels.data(), 6, first, 2, LT_DTYPE_BF16, 2048, 3, bf, kg) == 0) ++bad;
    if (lt_adamw_fp32_workspace_bytes(6) == 0 || lt_grad_sqnorm_partials_workspace_bytes(6) == 0 ||
        lt_grad_sqnorm_finish_workspace_bytes(6) == 0) ++bad;
    // argument errors are reported before any device call
    float* p[1] = {nullptr};
    const void* g[1] = {nullptr};
    int8_t* mq[1] = {nullptr}; uint8_t* vq[1] = {nullptr}; float* a[1] = {nullptr};
    int64_t n1[1] = {16};
    if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, n1, 1, 2048, LT_MAP_LINEAR,
                                 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, nullptr, nullptr, nullptr, nullptr, 0, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, n1, 1, 1000, LT_MAP_LINEAR,
                                 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, nullptr, nullptr, nullptr, nullptr, 0, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, n1, 1, 2048, 7,
                                 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, nullptr, nullptr, nullptr, nullptr, 0, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    if (lt_grad_sqnorm(g, n1, 1, 9, nullptr, 0, nullptr, nullptr, nullptr, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    if (lt_clip_coef(nullptr, 1.0f, nullptr, nullptr, nullptr, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    // eps must be > 0, also in fp32 (checked before any pointer or device call)
    for (double bad_eps : {0.0, -1e-8, 1e-50, (double)INFINITY})
        if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, n1, 1, 2048,
                                     LT_MAP_LINEAR, 1e-4, 0.9, 0.999, bad_eps, 0.01, 1, nullptr,
                                     nullptr, nullptr, nullptr, 0, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    // block sizes: multiples of 64 in [64, 65536]
    for (int bad_block : {0, 32, 96 + 8, 65536 + 64})
        if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, n1, 1, bad_block,
                                     LT_MAP_LINEAR, 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, nullptr,
                                     nullptr, nullptr, nullptr, 0, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    if (lt_adamw_fp32_step(p, g, LT_DTYPE_F32, p, p, nullptr, n1, 1, NAN, 0.9, 0.999, 1e-8, 0.01, 1,
                           nullptr, nullptr, nullptr, nullptr, 0, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    // empty lists and zero-element tensors: validated, then nothing to launch
    alignas(256) static uint8_t host_ws[4096];
    if (lt_workspace_release(nullptr) != LT_OK || lt_workspace_release(host_ws) != LT_OK) ++bad;
    if (lt_select_8bit_slice(nullptr, 0, 0.5, nullptr, &chosen) != LT_OK || chosen != 0) ++bad;
    if (lt_hybrid8bit_adamw_step(nullptr, nullptr, LT_DTYPE_BF16, nullptr, nullptr, nullptr, nullptr,
                                 nullptr, nullptr, 0, 2048, LT_MAP_LINEAR, 1e-4, 0.9, 0.999, 1e-8,
                                 0.01, 1, nullptr, nullptr, nullptr, host_ws, sizeof host_ws, nullptr) != LT_OK) ++bad;
    int64_t n0[2] = {0, 0};
    if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, n0, 1, 2048, LT_MAP_DYNAMIC,
                                 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, nullptr, nullptr, nullptr, host_ws,
                                 sizeof host_ws, nullptr) != LT_OK) ++bad;
    if (lt_adamw_fp32_step(nullptr, nullptr, LT_DTYPE_F32, nullptr, nullptr, nullptr, nullptr, 0, 1e-4,
                           0.9, 0.999, 1e-8, 0.01, 1, nullptr, nullptr, nullptr, host_ws, sizeof host_ws,
                           nullptr) != LT_OK) ++bad;
    const void* g2[2] = {nullptr, nullptr};  // pointers of empty tensors are not read
    if (lt_grad_sqnorm_partials(g2, n0, 2, LT_DTYPE_BF16, nullptr, nullptr, 0, nullptr) != LT_OK) ++bad;
    if (lt_grad_sqnorm_partials(nullptr, n0, 2, LT_DTYPE_BF16, nullptr, nullptr, 0, nullptr) !=
        LT_ERR_INVALID_ARG) ++bad;  // a NULL list of two tensors
    int64_t nneg[1] = {-1};
    if (lt_hybrid8bit_adamw_step(p, g, LT_DTYPE_BF16, mq, a, vq, a, nullptr, nneg, 1, 2048, LT_MAP_LINEAR,
                                 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, nullptr, nullptr, nullptr, host_ws,
                                 sizeof host_ws, nullptr) != LT_ERR_INVALID_ARG) ++bad;
    if (lt_grad_chunk_count(n0, 2) != 0 || lt_grad_sqnorm_workspace_bytes(nullptr, 0) == 0) ++bad;
    // overlap rule: the addresses are compared before anything is read or launched
    // (a host buffer stands in for device memory; no workspace, so a call that
    // passes the overlap check stops at the workspace check)
    alignas(256) static uint8_t mem[1 << 16];
    int64_t n2[2] = {1024, 1024};
    float* pw[2] = {(float*)(mem), (float*)(mem + 4096)};
    const void* gw[2] = {mem + 8192, mem + 8192};  // one gradient for both: only read
    int8_t* mqw[2] = {(int8_t*)(mem + 12288), (int8_t*)(mem + 13312)};
    uint8_t* vqw[2] = {mem + 14336, mem + 15360};
    float* maw[2] = {(float*)(mem + 16384), (float*)(mem + 16388)};
    float* vaw[2] = {(float*)(mem + 16392), (float*)(mem + 16396)};
    auto step8 = [&]() {
        return lt_hybrid8bit_adamw_step(pw, gw, LT_DTYPE_BF16, mqw, maw, vqw, vaw, nullptr, n2, 2,
                                        2048, LT_MAP_LINEAR, 1e-4, 0.9, 0.999, 1e-8, 0.01, 1,
                                        nullptr, nullptr, nullptr, nullptr, 0, nullptr);
    };
    if (step8() != LT_ERR_WORKSPACE) ++bad;       // disjoint, shared gradient
    pw[1] = (float*)(mem + 4080);                 // params[1] shares the last 16 bytes of params[0]
    if (step8() != LT_ERR_INVALID_ARG) ++bad;
    pw[1] = (float*)(mem + 4096);
    vaw[1] = (float*)(mem + 8192 + 2044);         // a v scale inside the gradient
    if (step8() != LT_ERR_INVALID_ARG) ++bad;
    vaw[1] = (float*)(mem + 16396);
    mqw[1] = (int8_t*)(mem + 12288);              // m codes of both tensors at one address
    if (step8() != LT_ERR_INVALID_ARG) ++bad;
    mqw[1] = (int8_t*)(mem + 13312);
    if (step8() != LT_ERR_WORKSPACE) ++bad;
    float* ea[2] = {(float*)(mem + 20480), (float*)(mem + 24576)};
    float* es[2] = {(float*)(mem + 28672), (float*)(mem + 32768)};
    auto step32 = [&]() {
        return lt_adamw_fp32_step(pw, gw, LT_DTYPE_BF16, ea, es, nullptr, n2, 2, 1e-4, 0.9, 0.999,
                                  1e-8, 0.01, 1, nullptr, nullptr, nullptr, nullptr, 0, nullptr);
    };
    if (step32() != LT_ERR_WORKSPACE) ++bad;
    es[0] = (float*)(mem + 24576 + 4080);         // exp_avg_sq[0] shares 16 bytes with exp_avg[1]
    if (step32() != LT_ERR_INVALID_ARG) ++bad;
    // streamed step: a workspace sized for resident gradients is too small for the
    // ring that carries them (3 slots of a 2-tensor layer), which the call reports
    // before it touches anything
    {
        int64_t sn[2] = {1024, 1024};
        int lf[2] = {0, 2};
        const size_t kept = lt_streamed_workspace_bytes(sn, 2, lf, 1, LT_DTYPE_BF16, 2048, 3, 0, 1);
        const size_t twice = lt_streamed_workspace_bytes(sn, 2, lf, 1, LT_DTYPE_BF16, 2048, 3, 0, 0);
        if (!(kept > 0 && twice > kept)) ++bad;
        static double dS; static float dc, dn; static int32_t dst;
        for (int keep = 0; keep < 2; ++keep) {
            const lt_err e = lt_streamed_hybrid8bit_adamw_step(
                pw, gw, LT_DTYPE_BF16, mqw, maw, vqw, vaw, nullptr, sn, 2, lf, 1, 2048,
                LT_MAP_LINEAR, 1e-4, 0.9, 0.999, 1e-8, 0.01, 1, 1.0f, 0, keep, 3, mem,
                keep ? kept - 256 : kept, &dS, &dn, &dc, &dst, nullptr, nullptr, nullptr, nullptr);
            if (e != LT_ERR_WORKSPACE) ++bad;
        }
    }
    if (lt_last_error() == nullptr || lt_last_error()[0] == 0) ++bad;
    printf("host checks: %d failures; last error: %s\n", bad, lt_last_error());
    return bad != 0;
}
