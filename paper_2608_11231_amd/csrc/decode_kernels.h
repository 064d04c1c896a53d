// Host-side launcher of the decode-step kernel.
#pragma once
#include "lkv_device.h"

namespace lkv {

struct DecodeArgs {
    int32_t n_req, h_qk, h_v, dv;
    int32_t io_bf16, gate_bf16;
    const void* q;     // GDN q | SSD C   [n_req, h_qk, dk]
    const void* k;     // GDN k | SSD B   [n_req, h_qk, dk]
    const void* v;     // GDN v | SSD x   [n_req, h_v, dv]
    const void* g;     // GDN log(alpha) [n_req, h_v] | SSD dt [n_req, H] f32
    const void* beta;  // GDN beta [n_req, h_v]       | SSD unused
    const float* A;    // SSD A [H]
    float scale;
    float* S;          // [n_req, h_v, dv, dk] f32, updated in place
    void* out;         // [n_req, h_v, dv] io dtype, or null
};

hipError_t launch_decode(int family, int dk, const DecodeArgs& a, hipStream_t st);

}  // namespace lkv
