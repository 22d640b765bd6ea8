// Internal interface between the C ABI (attn_api.cpp) and the HIP kernels.
//
// A "segment" is one batch entry (fixed length) or one packed sequence.  Row i
// of head h of segment z of a q-like tensor (q, o, dO, dq; Hq heads) is at
//   base + start * row_stride + z * batch_stride + h * head_stride
//        + i * row_stride                                    (elements)
// where start = cu[z] and batch_stride = 0 for packed input, and start = 0
// for fixed-length input;
// k-like tensors (k, v, dk, dv; Hkv heads) use the kv strides.  Row-indexed
// fp32 arrays (lse, Delta) follow the same rule with their own strides and a
// unit row stride.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

struct Layout {
  const int* cu;           // packed: cu_seqlens (device); fixed: nullptr
  int S;                   // fixed: sequence length; packed: max_seqlen
  int total;               // packed: T (rows); fixed: unused
  int nseg;                // B or nseq
  int Hq, Hkv, group;      // group = Hq / Hkv
  int64_t q_batch, q_head, q_row;     // strides of q-like tensors
  int64_t kv_batch, kv_head, kv_row;  // strides of k-like tensors
  int64_t r_batch, r_head;            // strides of lse / Delta (row stride 1)
};

struct FwdArgs {
  Layout L;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  float scale_log2;        // softmax scale * log2(e)
  int causal;
};

struct BwdArgs {
  Layout L;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const float* lse;
  const uint16_t* dout;
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  float* delta;            // workspace: Delta, same layout as lse
  float* lse2;             // workspace: lse * log2(e), same layout as lse
  float scale;             // softmax scale
  float scale_log2;        // scale * log2(e)
  int causal;
};

// Launchers: enqueue on `stream`, return the hipGetLastError() of the launch.
hipError_t launch_fwd(const FwdArgs& a, int D, hipStream_t stream);
// phases: bit 0 = Delta and dQ kernel, bit 1 = dK/dV kernel.
hipError_t launch_bwd(const BwdArgs& a, int D, int phases, hipStream_t stream);

}  // namespace attn
