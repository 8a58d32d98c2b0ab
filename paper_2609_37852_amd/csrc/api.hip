// Host implementation of the C ABI (include/attn_fp8.h): argument checks,
// workspace layout and launch sequencing.  No device memory is allocated here.
#include <cmath>
#include <cstdio>
#include <cstdarg>
#include <mutex>
#include <string>

#include "attn_fp8.h"
#include "kernels.hpp"

// Scratch of attn_fp8_bwd_noalloc: device memory the library holds for the
// whole process on every device it runs on (one copy per device, each at its
// own address).  Host code never uses the array's name as an address: the
// device address of each device's copy is looked up once, with that device
// current, and kept in g_scratch_ptr below.
constexpr size_t kNoAllocScratchBytes = ATTN_FP8_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {

thread_local std::string g_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}

int ok() {
  g_error.clear();
  return ATTN_FP8_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int dtype_size(int dt) { return dt == ATTN_FP8_DTYPE_F32 ? 4 : dt == ATTN_FP8_DTYPE_BF16 ? 2 : 0; }

bool head_dim_ok(int64_t d) { return d == 64 || d == 128 || d == 192 || d == 256; }

bool pair_ok(int64_t dqk, int64_t dv) {
  return (dqk == 64 && dv == 64) || (dqk == 128 && dv == 128) || (dqk == 256 && dv == 256) ||
         (dqk == 192 && dv == 128);
}

// strides {b, n, h} of a [B, N, H, D] tensor with contiguous channels
int check_strides(const char* name, const int64_t* s, int esize) {
  if (!s) return fail(ATTN_FP8_EINVAL, "%s: strides pointer is NULL", name);
  for (int i = 0; i < 3; i++) {
    if (s[i] < 0) return fail(ATTN_FP8_EINVAL, "%s: negative stride %lld", name, (long long)s[i]);
    if ((s[i] * esize) % 16 != 0)
      return fail(ATTN_FP8_EALIGN, "%s: stride %lld elements is not a multiple of 16 bytes", name,
                  (long long)s[i]);
  }
  return ATTN_FP8_OK;
}

int check_ptr(const char* name, const void* p) {
  if (!p) return fail(ATTN_FP8_EINVAL, "%s is NULL", name);
  if (!aligned16(p)) return fail(ATTN_FP8_EALIGN, "%s is not 16-byte aligned", name);
  return ATTN_FP8_OK;
}

int check_mx(const char* name, const attn_fp8_mx* m, bool row, bool col) {
  if (!m) return fail(ATTN_FP8_EINVAL, "%s: operand pointer is NULL", name);
  std::string n(name);
  int rc;
  if (row) {
    if ((rc = check_ptr((n + ".code_row").c_str(), m->code_row))) return rc;
    if ((rc = check_ptr((n + ".scale_row").c_str(), m->scale_row))) return rc;
  }
  if (col) {
    if ((rc = check_ptr((n + ".code_col").c_str(), m->code_col))) return rc;
    if ((rc = check_ptr((n + ".scale_col").c_str(), m->scale_col))) return rc;
  }
  return ATTN_FP8_OK;
}

int64_t kv_len(const attn_fp8_problem* p) { return p->seqlen_kv ? p->seqlen_kv : p->seqlen; }

int check_problem(const attn_fp8_problem* p) {
  if (!p) return fail(ATTN_FP8_EINVAL, "problem is NULL");
  if (p->batch < 0 || p->seqlen < 0 || p->heads_q < 0 || p->heads_kv < 0)
    return fail(ATTN_FP8_EINVAL, "negative problem size");
  if (p->heads_kv == 0 && p->heads_q != 0) return fail(ATTN_FP8_EINVAL, "heads_kv is 0");
  if (p->heads_kv > 0 && p->heads_q % p->heads_kv != 0)
    return fail(ATTN_FP8_EUNSUPPORTED, "heads_q (%lld) is not a multiple of heads_kv (%lld)",
                (long long)p->heads_q, (long long)p->heads_kv);
  if (!pair_ok(p->dim_qk, p->dim_v))
    return fail(ATTN_FP8_EUNSUPPORTED, "head dims (%lld, %lld) not instantiated", (long long)p->dim_qk,
                (long long)p->dim_v);
  if (p->causal != 0 && p->causal != 1) return fail(ATTN_FP8_EINVAL, "causal must be 0 or 1");
  if (p->flags & ~(ATTN_FP8_FLAG_PBWD_BLOCK_SCALED | ATTN_FP8_FLAG_PROTECTED_DP | ATTN_FP8_FLAG_ISOLATE3))
    return fail(ATTN_FP8_EINVAL, "unknown flags 0x%x", p->flags);
  if ((p->flags & ATTN_FP8_FLAG_ISOLATE3) &&
      (p->flags & (ATTN_FP8_FLAG_PBWD_BLOCK_SCALED | ATTN_FP8_FLAG_PROTECTED_DP)))
    return fail(ATTN_FP8_EUNSUPPORTED, "three isolated channels with another numerics variant");
  if (p->flags & ATTN_FP8_FLAG_PROTECTED_DP) {
    if (p->flags & ATTN_FP8_FLAG_PBWD_BLOCK_SCALED)
      return fail(ATTN_FP8_EUNSUPPORTED, "protected dP with the block-scaled backward probability operand");
    if (p->dim_qk == 256 && p->dim_v == 256)
      return fail(ATTN_FP8_EUNSUPPORTED, "protected dP at head dims (256, 256) (its BF16 tiles exceed the LDS)");
  }
  if (p->seqlen_kv < 0) return fail(ATTN_FP8_EINVAL, "negative seqlen_kv");
  if (p->causal && p->seqlens_kv)
    return fail(ATTN_FP8_EINVAL, "seqlens_kv with the causal mask (the key length is the query length)");
  if ((reinterpret_cast<uintptr_t>(p->seqlens_q) | reinterpret_cast<uintptr_t>(p->seqlens_kv)) & 3u)
    return fail(ATTN_FP8_EALIGN, "seqlens_q / seqlens_kv not 4-byte aligned");
  const int64_t nk = kv_len(p);
  if (p->causal && nk != p->seqlen)
    return fail(ATTN_FP8_EUNSUPPORTED, "causal attention needs seqlen_kv == seqlen (%lld != %lld)", (long long)nk,
                (long long)p->seqlen);
  if (p->seqlen == 0 && nk != 0)
    return fail(ATTN_FP8_EUNSUPPORTED, "seqlen 0 with seqlen_kv %lld (no queries, keys without gradient)",
                (long long)nk);
  if (p->seqlen % 32 != 0 || nk % 32 != 0)
    return fail(ATTN_FP8_EUNSUPPORTED, "seqlen %lld / seqlen_kv %lld is not a multiple of 32", (long long)p->seqlen,
                (long long)nk);
  if (!(std::isfinite(p->softmax_scale) && p->softmax_scale > 0.f))
    return fail(ATTN_FP8_EINVAL, "softmax_scale must be finite and positive");
  if (p->batch > 65535 || p->heads_q > 65535 || p->seqlen > (int64_t(1) << 30) || nk > (int64_t(1) << 30))
    return fail(ATTN_FP8_EUNSUPPORTED, "problem exceeds the launch grid limits");
  // one launch dimension holds at most 2^32 - 1 work-items: the query-major
  // kernels launch 2 B Hq N of them, the backward 4 B Hkv Nk
  if (p->batch * p->heads_q * p->seqlen >= (int64_t(1) << 31) || p->batch * p->heads_kv * nk >= (int64_t(1) << 30))
    return fail(ATTN_FP8_EUNSUPPORTED, "problem exceeds the launch grid limits (B Hq N = %lld, B Hkv Nk = %lld)",
                (long long)(p->batch * p->heads_q * p->seqlen), (long long)(p->batch * p->heads_kv * nk));
  // the kernels address the operands of one GQA group (G = Hq / Hkv adjacent
  // heads) and one KV head with 32-bit buffer offsets
  if (p->heads_kv > 0) {
    const int64_t G = p->heads_q / p->heads_kv, D = p->dim_qk > p->dim_v ? p->dim_qk : p->dim_v;
    const int64_t L = G * p->seqlen > nk ? G * p->seqlen : nk;
    if (L * D >= (int64_t(1) << 32))
      return fail(ATTN_FP8_EUNSUPPORTED, "problem exceeds the 32-bit buffer offsets (max(G N, Nk) D = %lld)",
                  (long long)(L * D));
    // protected dP: the group's BF16 dO rows take 2 bytes per element
    if ((p->flags & ATTN_FP8_FLAG_PROTECTED_DP) && G * p->seqlen * p->dim_v * 2 >= (int64_t(1) << 32))
      return fail(ATTN_FP8_EUNSUPPORTED, "protected dP: the BF16 dO of one group exceeds 32-bit buffer offsets");
  }
  return ATTN_FP8_OK;
}


bool empty(const attn_fp8_problem* p) { return p->batch == 0 || p->seqlen == 0 || p->heads_q == 0; }

afp8::AttnArgs base_args(const attn_fp8_problem* p) {
  afp8::AttnArgs a{};
  a.B = p->batch;
  a.N = p->seqlen;
  a.Hq = p->heads_q;
  a.Hkv = p->heads_kv;
  a.G = p->heads_q / p->heads_kv;
  a.Nk = kv_len(p);
  a.causal = p->causal;
  a.pmx = (p->flags & ATTN_FP8_FLAG_PBWD_BLOCK_SCALED) != 0;
  a.iso3 = (p->flags & ATTN_FP8_FLAG_ISOLATE3) != 0;
  a.lens_q = p->seqlens_q;
  a.lens_k = p->causal ? nullptr : p->seqlens_kv;
  a.cast_dump = p->cast_dump;
  a.tau = p->softmax_scale;
  a.c = (float)((double)p->softmax_scale * 1.4426950408889634);
  return a;
}

// Per-channel maxima of Q and K enable the isolated score channel.
void set_amax(afp8::AttnArgs& a, const attn_fp8_mx* q, const attn_fp8_mx* k) {
  const bool both = q && k && q->channel_amax && k->channel_amax;
  a.q_amax = both ? q->channel_amax : nullptr;
  a.k_amax = both ? k->channel_amax : nullptr;
}

void set_row(const attn_fp8_mx* m, const uint8_t*& code, const uint8_t*& scale) {
  code = m->code_row;
  scale = m->scale_row;
}
void set_col(const attn_fp8_mx* m, const uint8_t*& code, const uint8_t*& scale) {
  code = m->code_col;
  scale = m->scale_col;
}

size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

// stored dQ operand units (2048 B each) and their exponents (2 B each)
size_t units_per_head(const attn_fp8_problem* p) {
  return (size_t)afp8::dq_units_per_head(p->seqlen, kv_len(p), p->causal != 0);
}
size_t ws_units_bytes(const attn_fp8_problem* p) {
  return round256((size_t)p->batch * p->heads_q * units_per_head(p) * 2048);
}
size_t ws_exp_bytes(const attn_fp8_problem* p) {
  return round256((size_t)p->batch * p->heads_q * units_per_head(p) * 2);
}
size_t ws_delta_bytes(const attn_fp8_problem* p) {
  return round256((size_t)p->batch * p->heads_q * p->seqlen * 2 * sizeof(float));
}
size_t ws_rows_bytes(const attn_fp8_problem* p) {
  return round256((size_t)p->batch * p->heads_q * ((p->seqlen + 63) / 64) * 1024);
}
size_t ws_tile_cs_bytes(const attn_fp8_problem* p) {
  return round256((size_t)p->batch * p->heads_q * ((p->seqlen + 63) / 64) * 2 * (p->dim_qk + p->dim_v));
}
size_t ws_tile_kcs_bytes(const attn_fp8_problem* p) {
  return round256((size_t)p->batch * p->heads_kv * ((kv_len(p) + 63) / 64) * 2 * p->dim_qk);
}
// protected dP: BF16 copies of dO [B, Hq, N, Dv] and V [B, Hkv, Nk, Dv]
size_t ws_do_bf16_bytes(const attn_fp8_problem* p) {
  return (p->flags & ATTN_FP8_FLAG_PROTECTED_DP) ? round256((size_t)p->batch * p->heads_q * p->seqlen * p->dim_v * 2)
                                                 : 0;
}
size_t ws_v_bf16_bytes(const attn_fp8_problem* p) {
  return (p->flags & ATTN_FP8_FLAG_PROTECTED_DP) ? round256((size_t)p->batch * p->heads_kv * kv_len(p) * p->dim_v * 2)
                                                 : 0;
}
size_t ws_bwd_bytes(const attn_fp8_problem* p) {
  return ws_units_bytes(p) + ws_exp_bytes(p) + ws_delta_bytes(p) + ws_rows_bytes(p) + ws_tile_cs_bytes(p) +
         ws_tile_kcs_bytes(p) + ws_do_bf16_bytes(p) + ws_v_bf16_bytes(p);
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(ATTN_FP8_EHIP, "%s: %s", what, hipGetErrorString(e));
  return ATTN_FP8_OK;
}

int check_delta_inputs(const attn_fp8_problem* p, int mode, const attn_fp8_mx* q, const attn_fp8_mx* k,
                       const attn_fp8_mx* v, const attn_fp8_mx* dout, const float* lse, const void* dout_raw,
                       int dout_dtype, const int64_t* dout_strides, const void* o, int o_dtype,
                       const int64_t* o_strides) {
  int rc;
  if (mode == ATTN_FP8_DELTA_MATCHING || mode == ATTN_FP8_DELTA_MATCHING_COMPENSATED) {
    if (p->flags & ATTN_FP8_FLAG_PROTECTED_DP)
      return fail(ATTN_FP8_EUNSUPPORTED, "the matched correction of the protected-dP variant (its dP is BF16)");
    if ((p->flags & ATTN_FP8_FLAG_ISOLATE3) && mode == ATTN_FP8_DELTA_MATCHING_COMPENSATED)
      return fail(ATTN_FP8_EUNSUPPORTED, "the compensated correction with three isolated channels");
    if ((rc = check_mx("q", q, true, false)) || (rc = check_mx("k", k, true, false)) ||
        (rc = check_mx("v", v, true, false)) || (rc = check_mx("dout", dout, true, false)) ||
        (rc = check_ptr("lse", lse)))
      return rc;
  } else if (mode == ATTN_FP8_DELTA_STALE_ROWSUM) {
    if (!dtype_size(dout_dtype) || !dtype_size(o_dtype)) return fail(ATTN_FP8_EINVAL, "bad dout/o dtype");
    if ((rc = check_ptr("dout_raw", dout_raw)) || (rc = check_ptr("o", o)) ||
        (rc = check_strides("dout_raw", dout_strides, dtype_size(dout_dtype))) ||
        (rc = check_strides("o", o_strides, dtype_size(o_dtype))))
      return rc;
  } else if (mode == ATTN_FP8_DELTA_CONSISTENT_DO) {
    if (!dtype_size(o_dtype)) return fail(ATTN_FP8_EINVAL, "bad o dtype");
    if ((rc = check_mx("dout", dout, true, false)) || (rc = check_ptr("o", o)) ||
        (rc = check_strides("o", o_strides, dtype_size(o_dtype))))
      return rc;
  } else {
    return fail(ATTN_FP8_EINVAL, "unknown delta_mode %d", mode);
  }
  return ATTN_FP8_OK;
}

int launch_delta(const attn_fp8_problem* p, int mode, const attn_fp8_mx* q, const attn_fp8_mx* k,
                 const attn_fp8_mx* v, const attn_fp8_mx* dout, const float* lse, const void* dout_raw,
                 int dout_dtype, const int64_t* dout_strides, const void* o, int o_dtype,
                 const int64_t* o_strides, float* delta, hipStream_t stream) {
  if (mode == ATTN_FP8_DELTA_MATCHING || mode == ATTN_FP8_DELTA_MATCHING_COMPENSATED) {
    afp8::AttnArgs a = base_args(p);
    a.comp = mode == ATTN_FP8_DELTA_MATCHING_COMPENSATED;
    set_row(q, a.q_code, a.q_scale);
    set_row(k, a.k_code, a.k_scale);
    set_row(v, a.v_code, a.v_scale);
    set_row(dout, a.do_code, a.do_scale);
    set_amax(a, q, k);
    a.lse = lse;
    a.delta_out = delta;
    return hip_status(afp8::launch_delta_matching(a, (int)p->dim_qk, (int)p->dim_v, stream), "delta_matching");
  }
  afp8::StaleArgs s{};
  s.o = o;
  for (int i = 0; i < 3; i++) s.os[i] = o_strides[i];
  s.delta = delta;
  s.B = p->batch;
  s.N = p->seqlen;
  s.Hq = p->heads_q;
  s.Dv = (int)p->dim_v;
  s.lens_q = p->seqlens_q;
  s.lens_k = p->causal ? nullptr : p->seqlens_kv;
  s.Nk = kv_len(p);
  if (mode == ATTN_FP8_DELTA_CONSISTENT_DO) {
    s.do_code = dout->code_row;
    s.do_scale = dout->scale_row;
    return hip_status(afp8::launch_consistent_rowsum(s, o_dtype == ATTN_FP8_DTYPE_BF16, stream), "consistent_rowsum");
  }
  s.dout = dout_raw;
  for (int i = 0; i < 3; i++) s.ds[i] = dout_strides[i];
  return hip_status(afp8::launch_stale_rowsum(s, dout_dtype == ATTN_FP8_DTYPE_BF16, o_dtype == ATTN_FP8_DTYPE_BF16,
                                              stream),
                    "stale_rowsum");
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(ATTN_FP8_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(ATTN_FP8_EUNSUPPORTED, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(ATTN_FP8_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return ATTN_FP8_OK;
}

// Producer workspace: the key-mean partial sums (FP64 [B, H, N/32, D]) when
// centering, then the QK-normalization row scales (FP32 [B, N, H]) when a
// gain is given, each 256-byte aligned.
size_t align256(size_t n) { return (n + 255) & ~size_t(255); }
size_t ws_partials_bytes(int64_t B, int64_t N, int64_t H, int64_t D, const attn_fp8_producer* o) {
  return o->center ? align256(size_t(B * H * D * (N / 32)) * sizeof(double)) : 0;
}
size_t ws_rscale_bytes(int64_t B, int64_t N, int64_t H, const attn_fp8_producer* o) {
  return o->rms_gain ? align256(size_t(B * N * H) * sizeof(float)) : 0;
}

int check_producer(int64_t D, const attn_fp8_producer* o) {
  int rc;
  if (!o) return fail(ATTN_FP8_EINVAL, "producer options are NULL");
  if (!(std::isfinite(o->prescale) && o->prescale != 0.f))
    return fail(ATTN_FP8_EINVAL, "prescale must be finite and nonzero");
  if (o->center != 0 && o->center != 1) return fail(ATTN_FP8_EINVAL, "center = %d", (int)o->center);
  if (o->center && (rc = check_ptr("channel_mean", o->channel_mean))) return rc;
  if (o->rms_gain) {
    if (!(std::isfinite(o->rms_eps) && o->rms_eps >= 0.0)) return fail(ATTN_FP8_EINVAL, "rms_eps must be finite, >= 0");
    if (reinterpret_cast<uintptr_t>(o->rms_gain) & 15u) return fail(ATTN_FP8_EALIGN, "rms_gain is not 16-byte aligned");
  }
  if (o->rope_dim < 0 || o->rope_lo < 0) return fail(ATTN_FP8_EINVAL, "negative rope_lo / rope_dim");
  if (o->rope_dim > 0) {
    if (o->rope_dim % 32 != 0 || o->rope_lo % 32 != 0 || o->rope_lo + o->rope_dim > D)
      return fail(ATTN_FP8_EUNSUPPORTED, "rotary channels [%lld, %lld) are not 32-aligned inside D = %lld",
                  (long long)o->rope_lo, (long long)(o->rope_lo + o->rope_dim), (long long)D);
    if ((rc = check_ptr("rope_cs", o->rope_cs))) return rc;
  }
  if (o->seqlens && (reinterpret_cast<uintptr_t>(o->seqlens) & 3u))
    return fail(ATTN_FP8_EALIGN, "producer seqlens not 4-byte aligned");
  return ATTN_FP8_OK;
}

// opt NULL: the plain quantizer
int quantize_impl(const void* x, int x_dtype, int64_t B, int64_t N, int64_t H, int64_t D, const int64_t strides[3],
                  const attn_fp8_producer* opt, void* workspace, size_t workspace_bytes, const attn_fp8_mx* out,
                  int which, uint32_t* nonfinite_count, hipStream_t stream) {
  int rc;
  const int es = dtype_size(x_dtype);
  if (!es) return fail(ATTN_FP8_EINVAL, "x_dtype %d is not F32 or BF16", x_dtype);
  if (B < 0 || N < 0 || H < 0) return fail(ATTN_FP8_EINVAL, "negative size");
  if (!head_dim_ok(D)) return fail(ATTN_FP8_EUNSUPPORTED, "D = %lld not in {64,128,192,256}", (long long)D);
  if (N % 32 != 0) return fail(ATTN_FP8_EUNSUPPORTED, "N = %lld is not a multiple of 32", (long long)N);
  if (which < 1 || which > 3) return fail(ATTN_FP8_EINVAL, "which = %d", which);
  if (B > 65535 || H > 65535 || N > (int64_t(1) << 30)) return fail(ATTN_FP8_EUNSUPPORTED, "grid limits");
  if (opt && (rc = check_producer(D, opt))) return rc;
  if (opt && opt->rms_gain && B * N * H >= (int64_t(1) << 38))
    return fail(ATTN_FP8_EUNSUPPORTED, "grid limits (B N H = %lld rows for the norm)", (long long)(B * N * H));
  if (B == 0 || N == 0 || H == 0) return ok();  // empty: nothing is read or written
  if ((rc = check_ptr("x", x)) || (rc = check_strides("x", strides, es)) ||
      (rc = check_mx("out", out, which & 1, which & 2)))
    return rc;
  if (out->channel_amax) {
    if (!(which & 2)) return fail(ATTN_FP8_EINVAL, "channel_amax needs the col copy (which & COL)");
    if ((rc = check_ptr("out.channel_amax", out->channel_amax))) return rc;
  }
  afp8::QuantArgs a{};
  a.x = x;
  a.sb = strides[0];
  a.sn = strides[1];
  a.sh = strides[2];
  a.B = B;
  a.N = N;
  a.H = H;
  a.code_row = out->code_row;
  a.scale_row = out->scale_row;
  a.code_col = out->code_col;
  a.scale_col = out->scale_col;
  a.which = which;
  a.nonfinite = nonfinite_count;
  a.chan_amax = out->channel_amax;
  a.prescale = 1.0f;
  if (opt) {
    const size_t np = ws_partials_bytes(B, N, H, D, opt), need = np + ws_rscale_bytes(B, N, H, opt);
    if (need) {
      if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return fail(ATTN_FP8_EWORKSPACE, "workspace is NULL or not 256-byte aligned");
      if (workspace_bytes < need)
        return fail(ATTN_FP8_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
    }
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
    a.prescale = opt->prescale;
    if (opt->center) {
      a.mean = opt->channel_mean;
      a.partials = reinterpret_cast<double*>(ws);
      a.lens = opt->seqlens;
    }
    if (opt->rms_gain) {
      a.gain = opt->rms_gain;
      a.eps = (double)opt->rms_eps;
      a.rscale = reinterpret_cast<float*>(ws + np);
    }
    if (opt->rope_dim > 0) {
      a.rope = opt->rope_cs;
      a.rope_lo = (int)opt->rope_lo;
      a.rope_dim = (int)opt->rope_dim;
    }
  }
  if ((rc = hip_status(afp8::launch_quantize(a, (int)D, x_dtype == ATTN_FP8_DTYPE_BF16, stream), "quantize")))
    return rc;
  return ok();
}

}  // namespace

extern "C" {

const char* attn_fp8_last_error(void) { return g_error.c_str(); }

int attn_fp8_quantize(const void* x, int x_dtype, int64_t B, int64_t N, int64_t H, int64_t D,
                      const int64_t strides[3], const attn_fp8_mx* out, int which, uint32_t* nonfinite_count,
                      hipStream_t stream) {
  return quantize_impl(x, x_dtype, B, N, H, D, strides, nullptr, nullptr, 0, out, which, nonfinite_count, stream);
}

int attn_fp8_producer_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D, const attn_fp8_producer* opt,
                                     size_t* bytes) {
  int rc;
  if (!bytes) return fail(ATTN_FP8_EINVAL, "bytes is NULL");
  if (B < 0 || N < 0 || H < 0) return fail(ATTN_FP8_EINVAL, "negative size");
  if (!head_dim_ok(D)) return fail(ATTN_FP8_EUNSUPPORTED, "D = %lld not in {64,128,192,256}", (long long)D);
  if (N % 32 != 0) return fail(ATTN_FP8_EUNSUPPORTED, "N = %lld is not a multiple of 32", (long long)N);
  if (B > 65535 || H > 65535 || N > (int64_t(1) << 30)) return fail(ATTN_FP8_EUNSUPPORTED, "grid limits");
  if ((rc = check_producer(D, opt))) return rc;
  *bytes = ws_partials_bytes(B, N, H, D, opt) + ws_rscale_bytes(B, N, H, opt);
  return ok();
}

int attn_fp8_quantize_producer(const void* x, int x_dtype, int64_t B, int64_t N, int64_t H, int64_t D,
                               const int64_t strides[3], const attn_fp8_producer* opt, void* workspace,
                               size_t workspace_bytes, const attn_fp8_mx* out, int which, uint32_t* nonfinite_count,
                               hipStream_t stream) {
  if (!opt) return fail(ATTN_FP8_EINVAL, "producer options are NULL");
  return quantize_impl(x, x_dtype, B, N, H, D, strides, opt, workspace, workspace_bytes, out, which,
                       nonfinite_count, stream);
}

int attn_fp8_fwd(const attn_fp8_problem* p, const attn_fp8_mx* q, const attn_fp8_mx* k, const attn_fp8_mx* v,
                 void* o, int o_dtype, const int64_t o_strides[3], float* lse, hipStream_t stream) {
  int rc;
  if ((rc = check_problem(p))) return rc;
  if (!dtype_size(o_dtype)) return fail(ATTN_FP8_EINVAL, "o_dtype %d", o_dtype);
  if (empty(p)) return ok();
  if ((rc = check_mx("q", q, true, false)) || (rc = check_mx("k", k, true, false)) ||
      (rc = check_mx("v", v, false, true)) || (rc = check_ptr("o", o)) ||
      (rc = check_strides("o", o_strides, dtype_size(o_dtype))) || (rc = check_ptr("lse", lse)))
    return rc;
  afp8::AttnArgs a = base_args(p);
  set_row(q, a.q_code, a.q_scale);
  set_row(k, a.k_code, a.k_scale);
  set_col(v, a.vc_code, a.vc_scale);
  set_amax(a, q, k);
  a.o = o;
  for (int i = 0; i < 3; i++) a.os[i] = o_strides[i];
  a.o_bf16 = o_dtype == ATTN_FP8_DTYPE_BF16;
  a.lse_out = lse;
  if ((rc = hip_status(afp8::launch_fwd(a, (int)p->dim_qk, (int)p->dim_v, stream), "fwd"))) return rc;
  return ok();
}

int attn_fp8_delta(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q, const attn_fp8_mx* k,
                   const attn_fp8_mx* v, const attn_fp8_mx* dout, const float* lse, const void* dout_raw,
                   int dout_dtype, const int64_t dout_strides[3], const void* o, int o_dtype,
                   const int64_t o_strides[3], float* delta, hipStream_t stream) {
  int rc;
  if ((rc = check_problem(p))) return rc;
  if (delta_mode < ATTN_FP8_DELTA_MATCHING || delta_mode > ATTN_FP8_DELTA_MATCHING_COMPENSATED)
    return fail(ATTN_FP8_EINVAL, "unknown delta_mode %d", delta_mode);
  if (empty(p)) return ok();
  if ((rc = check_delta_inputs(p, delta_mode, q, k, v, dout, lse, dout_raw, dout_dtype, dout_strides, o, o_dtype,
                               o_strides)) ||
      (rc = check_ptr("delta", delta)))
    return rc;
  if ((rc = launch_delta(p, delta_mode, q, k, v, dout, lse, dout_raw, dout_dtype, dout_strides, o, o_dtype,
                         o_strides, delta, stream)))
    return rc;
  return ok();
}

int attn_fp8_bwd_workspace_size(const attn_fp8_problem* p, size_t* bytes) {
  int rc;
  if ((rc = check_problem(p))) return rc;
  if (!bytes) return fail(ATTN_FP8_EINVAL, "bytes is NULL");
  *bytes = ws_bwd_bytes(p);
  return ok();
}

// The backward, FP8 dP (v_raw NULL) or protected dP (dP = dO V^T from BF16
// copies of dout_raw and v_raw packed into the workspace).
static int bwd_impl(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q, const attn_fp8_mx* k,
                    const attn_fp8_mx* v, const attn_fp8_mx* dout, const float* lse, const void* dout_raw,
                    int dout_dtype, const int64_t dout_strides[3], const void* v_raw, int v_dtype,
                    const int64_t v_strides[3], const void* o, int o_dtype, const int64_t o_strides[3],
                    const float* delta_in, void* dq, void* dk, void* dv, int grad_dtype,
                    const int64_t dq_strides[3], const int64_t dk_strides[3], const int64_t dv_strides[3],
                    void* workspace, size_t workspace_bytes, double* rowstats, const hipEvent_t* main_events,
                    hipStream_t stream) {
  int rc;
  const bool pdp = v_raw != nullptr;
  if ((rc = check_problem(p))) return rc;
  if (delta_mode < ATTN_FP8_DELTA_MATCHING || delta_mode > ATTN_FP8_DELTA_MATCHING_COMPENSATED)
    return fail(ATTN_FP8_EINVAL, "unknown delta_mode %d", delta_mode);
  if ((p->flags & ATTN_FP8_FLAG_ISOLATE3) && delta_mode == ATTN_FP8_DELTA_MATCHING_COMPENSATED)
    return fail(ATTN_FP8_EUNSUPPORTED, "the compensated correction with three isolated channels");
  const int gs = dtype_size(grad_dtype);
  if (!gs) return fail(ATTN_FP8_EINVAL, "grad_dtype %d", grad_dtype);
  if (empty(p)) return ok();
  if ((rc = check_mx("q", q, true, true)) || (rc = check_mx("k", k, true, true)) ||
      (!pdp && (rc = check_mx("v", v, true, false))) || (rc = check_mx("dout", dout, !pdp, true)) ||
      (rc = check_ptr("lse", lse)) || (rc = check_ptr("dq", dq)) || (rc = check_ptr("dk", dk)) ||
      (rc = check_ptr("dv", dv)) || (rc = check_strides("dq", dq_strides, gs)) ||
      (rc = check_strides("dk", dk_strides, gs)) || (rc = check_strides("dv", dv_strides, gs)))
    return rc;
  if (pdp) {
    if (!dtype_size(dout_dtype) || !dtype_size(v_dtype)) return fail(ATTN_FP8_EINVAL, "bad dout_raw / v_raw dtype");
    if ((rc = check_ptr("dout_raw", dout_raw)) || (rc = check_strides("dout_raw", dout_strides, dtype_size(dout_dtype))) ||
        (rc = check_strides("v_raw", v_strides, dtype_size(v_dtype))))
      return rc;
  }
  if (delta_in) {
    if ((rc = check_ptr("delta_in", delta_in))) return rc;
  } else if ((rc = check_delta_inputs(p, delta_mode, q, k, v, dout, lse, dout_raw, dout_dtype, dout_strides, o,
                                      o_dtype, o_strides))) {
    return rc;
  }
  if (rowstats && !aligned16(rowstats)) return fail(ATTN_FP8_EALIGN, "rowstats is not 16-byte aligned");
  if (p->cast_dump && !rowstats) return fail(ATTN_FP8_EINVAL, "cast_dump without rowstats");
  if (p->cast_dump && !aligned16(p->cast_dump)) return fail(ATTN_FP8_EALIGN, "cast_dump is not 16-byte aligned");
  const size_t need = ws_bwd_bytes(p);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(ATTN_FP8_EWORKSPACE, "workspace is NULL or not 256-byte aligned");
  if (workspace_bytes < need)
    return fail(ATTN_FP8_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);

  uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);
  uint8_t* ds_units = ws;
  uint8_t* ds_exp = ds_units + ws_units_bytes(p);
  float* delta = reinterpret_cast<float*>(ds_exp + ws_exp_bytes(p));
  float* rows = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(delta) + ws_delta_bytes(p));
  uint8_t* tile_cs = reinterpret_cast<uint8_t*>(rows) + ws_rows_bytes(p);
  uint8_t* tile_kcs = tile_cs + ws_tile_cs_bytes(p);
  uint16_t* do_bf16 = reinterpret_cast<uint16_t*>(tile_kcs + ws_tile_kcs_bytes(p));
  uint16_t* v_bf16 = reinterpret_cast<uint16_t*>(reinterpret_cast<uint8_t*>(do_bf16) + ws_do_bf16_bytes(p));
  if (delta_in) {
    delta = const_cast<float*>(delta_in);
  } else if ((rc = launch_delta(p, delta_mode, q, k, v, dout, lse, dout_raw, dout_dtype, dout_strides, o, o_dtype,
                                o_strides, delta, stream))) {
    return rc;
  }

  afp8::AttnArgs a = base_args(p);
  set_row(q, a.q_code, a.q_scale);
  set_row(k, a.k_code, a.k_scale);
  if (!pdp) {
    set_row(v, a.v_code, a.v_scale);
    set_row(dout, a.do_code, a.do_scale);
  }
  set_col(q, a.qc_code, a.qc_scale);
  set_col(k, a.kc_code, a.kc_scale);
  set_col(dout, a.doc_code, a.doc_scale);
  set_amax(a, q, k);
  a.lse = lse;
  a.delta = delta;
  a.ds_units = ds_units;
  a.ds_exp = ds_exp;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  for (int i = 0; i < 3; i++) {
    a.dks[i] = dk_strides[i];
    a.dvs[i] = dv_strides[i];
    a.dqs[i] = dq_strides[i];
  }
  a.grad_bf16 = grad_dtype == ATTN_FP8_DTYPE_BF16;
  a.comp = delta_mode == ATTN_FP8_DELTA_MATCHING_COMPENSATED;
  a.rowstats = rowstats;
  a.rows = rows;
  a.tile_cs = tile_cs;
  a.tile_kcs = tile_kcs;
  if (pdp) {
    a.pdp = 1;
    a.comp = 0;
    a.do_bf16 = do_bf16;
    a.v_bf16 = v_bf16;
    if ((rc = hip_status(afp8::launch_pack_bf16(dout_raw, dout_dtype == ATTN_FP8_DTYPE_BF16, dout_strides, p->batch,
                                                p->seqlen, p->heads_q, (int)p->dim_v, a.lens_q, do_bf16, stream),
                         "pack dO")) ||
        (rc = hip_status(afp8::launch_pack_bf16(v_raw, v_dtype == ATTN_FP8_DTYPE_BF16, v_strides, p->batch, kv_len(p),
                                                p->heads_kv, (int)p->dim_v, p->causal ? a.lens_q : a.lens_k, v_bf16,
                                                stream),
                         "pack V")))
      return rc;
  }
  if ((rc = hip_status(afp8::launch_bwd_prep(a, (int)p->dim_qk, (int)p->dim_v, stream), "bwd_prep"))) return rc;
  if (main_events && (rc = hip_status(hipEventRecord(main_events[0], stream), "event record"))) return rc;
  if ((rc = hip_status(afp8::launch_bwd(a, (int)p->dim_qk, (int)p->dim_v, stream), "bwd"))) return rc;
  if (main_events && (rc = hip_status(hipEventRecord(main_events[1], stream), "event record"))) return rc;

  if ((rc = hip_status(afp8::launch_dq(a, (int)p->dim_qk, stream), "dq"))) return rc;
  return ok();
}

int attn_fp8_bwd(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q, const attn_fp8_mx* k,
                 const attn_fp8_mx* v, const attn_fp8_mx* dout, const float* lse, const void* dout_raw,
                 int dout_dtype, const int64_t dout_strides[3], const void* o, int o_dtype,
                 const int64_t o_strides[3], const float* delta_in, void* dq, void* dk, void* dv, int grad_dtype,
                 const int64_t dq_strides[3], const int64_t dk_strides[3], const int64_t dv_strides[3],
                 void* workspace, size_t workspace_bytes, double* rowstats, const hipEvent_t* main_events,
                 hipStream_t stream) {
  if (p && (p->flags & ATTN_FP8_FLAG_PROTECTED_DP))
    return fail(ATTN_FP8_EINVAL, "a protected-dP problem takes attn_fp8_bwd_protected_dp (it reads the raw V)");
  return bwd_impl(p, delta_mode, q, k, v, dout, lse, dout_raw, dout_dtype, dout_strides, nullptr, 0, nullptr, o,
                  o_dtype, o_strides, delta_in, dq, dk, dv, grad_dtype, dq_strides, dk_strides, dv_strides, workspace,
                  workspace_bytes, rowstats, main_events, stream);
}

int attn_fp8_bwd_protected_dp(const attn_fp8_problem* p, const attn_fp8_mx* q, const attn_fp8_mx* k,
                              const attn_fp8_mx* dout, const float* lse, const void* dout_raw, int dout_dtype,
                              const int64_t dout_strides[3], const void* v_raw, int v_dtype,
                              const int64_t v_strides[3], const void* o, int o_dtype, const int64_t o_strides[3],
                              const float* delta_in, void* dq, void* dk, void* dv, int grad_dtype,
                              const int64_t dq_strides[3], const int64_t dk_strides[3],
                              const int64_t dv_strides[3], void* workspace, size_t workspace_bytes,
                              double* rowstats, hipStream_t stream) {
  int rc;
  if ((rc = check_problem(p))) return rc;
  if (!(p->flags & ATTN_FP8_FLAG_PROTECTED_DP))
    return fail(ATTN_FP8_EINVAL, "attn_fp8_bwd_protected_dp needs ATTN_FP8_FLAG_PROTECTED_DP in the problem's flags");
  if (empty(p)) return ok();
  if ((rc = check_ptr("v_raw", v_raw))) return rc;
  return bwd_impl(p, ATTN_FP8_DELTA_STALE_ROWSUM, q, k, nullptr, dout, lse, dout_raw, dout_dtype, dout_strides, v_raw,
                  v_dtype, v_strides, o, o_dtype, o_strides, delta_in, dq, dk, dv, grad_dtype, dq_strides, dk_strides,
                  dv_strides, workspace, workspace_bytes, rowstats, nullptr, stream);
}

int attn_fp8_bwd_noalloc(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q, const attn_fp8_mx* k,
                         const attn_fp8_mx* v, const attn_fp8_mx* dout, const float* lse, const void* dout_raw,
                         int dout_dtype, const int64_t dout_strides[3], const void* o, int o_dtype,
                         const int64_t o_strides[3], const float* delta_in, void* dq, void* dk, void* dv,
                         int grad_dtype, const int64_t dq_strides[3], const int64_t dk_strides[3],
                         const int64_t dv_strides[3], double* rowstats, const hipEvent_t* main_events,
                         hipStream_t stream) {
  int rc;
  if ((rc = check_problem(p))) return rc;
  if (p->flags & ATTN_FP8_FLAG_PROTECTED_DP)
    return fail(ATTN_FP8_EINVAL, "attn_fp8_bwd_noalloc runs the FP8-dP backward (no protected dP)");
  if (empty(p)) return ok();
  const size_t need = ws_bwd_bytes(p);
  if (need > kNoAllocScratchBytes)
    return fail(ATTN_FP8_EUNSUPPORTED,
                "attn_fp8_bwd_noalloc: this problem needs %zu bytes of scratch; the library's scratch holds %zu "
                "(use attn_fp8_bwd with a caller workspace)",
                need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if ((rc = scratch_address(&ws))) return rc;
  return attn_fp8_bwd(p, delta_mode, q, k, v, dout, lse, dout_raw, dout_dtype, dout_strides, o, o_dtype, o_strides,
                      delta_in, dq, dk, dv, grad_dtype, dq_strides, dk_strides, dv_strides, ws, kNoAllocScratchBytes,
                      rowstats, main_events, stream);
}

}  // extern "C"
