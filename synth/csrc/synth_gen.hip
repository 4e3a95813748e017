// Device twin of synth/gen.py: fills synthetic inputs in HBM with the same
// bits as the host generator.  Holds no arithmetic of the decode method.
//
// Every value is SplitMix64(key + (ctr + 1) * gamma) shaped into an
// Irwin-Hall(4) normal stand-in or a 24-bit uniform, with each floating-point
// step a single IEEE operation (__fmul_rn / __fadd_rn, no contraction), then
// rounded to bf16 by round-to-nearest-even when the workload stores bf16.
// Per-(kind, layer, seq) keys come precomputed from the host.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kM1 = 0xBF58476D1CE4E5B9ull;
constexpr uint64_t kM2 = 0x94D049BB133111EBull;
constexpr int kKinds = 12;
constexpr int kMaxFlat = 16;

// kinds, as in gen.py
constexpr int KIND_K = 1, KIND_V = 2, KIND_Q = 3, KIND_LOGIT = 4, KIND_HH = 5, KIND_BETA = 6,
              KIND_AXIS = 7, KIND_ALPHA = 8;

}  // namespace

struct SynthParams {
    const uint64_t* keys;      // [kKinds][L][B]; logits use layer 0
    const uint64_t* hh_thr;    // [B]
    int32_t L, B, Hq, Hkv, D, V;
    int32_t recipe;            // 0 gauss, 1 heavy hitters
    int32_t bf16;
    float ih_scale, sigma, flat_sigma;
    float beta_lo, beta_span, alpha_lo, alpha_span, nonhh_scale, q_noise;
    int32_t n_flat;
    int32_t flat[kMaxFlat];
};

namespace {

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * kM1;
    z = (z ^ (z >> 27)) * kM2;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t draw(uint64_t key, uint64_t ctr) {
    return mix64(key + (ctr + 1ull) * kGamma);
}

__device__ __forceinline__ float gauss(uint64_t z, float scale) {
    const int s = (int)(z & 0xFFFF) + (int)((z >> 16) & 0xFFFF) + (int)((z >> 32) & 0xFFFF) +
                  (int)(z >> 48);
    return __fmul_rn((float)(s - 131070), scale);
}

__device__ __forceinline__ float uniform24(uint64_t z) {
    return __fmul_rn((float)(uint32_t)(z >> 40), 0x1p-24f);
}

__device__ __forceinline__ uint16_t bf16_bits(float x) {
    const uint32_t b = __float_as_uint(x);
    return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ void store(void* out, size_t i, float x, int bf16) {
    if (bf16) reinterpret_cast<uint16_t*>(out)[i] = bf16_bits(x);
    else reinterpret_cast<float*>(out)[i] = x;
}

__device__ __forceinline__ uint64_t key_of(const SynthParams& w, int kind, int l, int b) {
    return w.keys[((size_t)kind * w.L + l) * w.B + b];
}

// value of K (is_v = 0) or V (is_v = 1) at (layer, seq, position, kv head, dim)
__device__ float kv_value(const SynthParams& w, int l, int b, uint64_t p, int g, int d, int is_v) {
    const uint64_t ctr = (p * (uint64_t)w.Hkv + g) * (uint64_t)w.D + d;
    const float z = gauss(draw(key_of(w, is_v ? KIND_V : KIND_K, l, b), ctr), w.ih_scale);
    if (is_v || w.recipe != 1) return z;
    const uint64_t ax = draw(key_of(w, KIND_AXIS, l, b), (uint64_t)g);
    if ((int)(ax % (uint64_t)w.D) != d) return z;
    const bool hh = (draw(key_of(w, KIND_HH, l, b), p) >> 11) < w.hh_thr[b];
    if (!hh) return __fmul_rn(z, w.nonhh_scale);
    const float u = uniform24(draw(key_of(w, KIND_BETA, l, b), p * (uint64_t)w.Hkv + g));
    const float beta = __fadd_rn(__fmul_rn(u, w.beta_span), w.beta_lo);
    return ((ax >> 32) & 1ull) ? -beta : beta;
}

__global__ void kv_kernel(SynthParams w, int l, int b, int64_t p0, int64_t n, void* K, void* V) {
    const size_t per = (size_t)w.Hkv * w.D;
    const size_t total = (size_t)n * per;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        const uint64_t p = (uint64_t)p0 + i / per;
        const int g = (int)((i % per) / w.D), d = (int)(i % w.D);
        store(K, i, kv_value(w, l, b, p, g, d, 0), w.bf16);
        store(V, i, kv_value(w, l, b, p, g, d, 1), w.bf16);
    }
}

// new-token rows of steps t0 .. t0+steps-1: out [steps][L][B][Hkv][D]
__global__ void new_kv_kernel(SynthParams w, int t0, int steps, const int32_t* plen, void* K, void* V) {
    const size_t per = (size_t)w.Hkv * w.D;
    const size_t total = (size_t)steps * w.L * w.B * per;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        size_t r = i / per;
        const int b = (int)(r % w.B); r /= w.B;
        const int l = (int)(r % w.L); r /= w.L;
        const int t = t0 + (int)r;
        const uint64_t p = (uint64_t)plen[b] + t - 1;
        const int g = (int)((i % per) / w.D), d = (int)(i % w.D);
        store(K, i, kv_value(w, l, b, p, g, d, 0), w.bf16);
        store(V, i, kv_value(w, l, b, p, g, d, 1), w.bf16);
    }
}

// queries of steps t0 .. t0+steps-1: out [steps][L][B][Hq][D]
__global__ void q_kernel(SynthParams w, int t0, int steps, void* Q) {
    const size_t per = (size_t)w.Hq * w.D;
    const size_t total = (size_t)steps * w.L * w.B * per;
    const int G = w.Hq / w.Hkv;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        size_t r = i / per;
        const int b = (int)(r % w.B); r /= w.B;
        const int l = (int)(r % w.L); r /= w.L;
        const uint64_t t = (uint64_t)(t0 + (int)r);
        const int h = (int)((i % per) / w.D), d = (int)(i % w.D);
        float q = gauss(draw(key_of(w, KIND_Q, l, b), t * per + (uint64_t)(h * w.D + d)), w.ih_scale);
        if (w.recipe == 1) {
            q = __fmul_rn(q, w.q_noise);
            const uint64_t ax = draw(key_of(w, KIND_AXIS, l, b), (uint64_t)(h / G));
            if ((int)(ax % (uint64_t)w.D) == d) {
                const float ua = uniform24(draw(key_of(w, KIND_ALPHA, l, b), t * w.Hq + h));
                const float alpha = __fadd_rn(__fmul_rn(ua, w.alpha_span), w.alpha_lo);
                q = __fadd_rn(q, ((ax >> 32) & 1ull) ? -alpha : alpha);
            }
        }
        store(Q, i, q, w.bf16);
    }
}

// logits after steps t0 .. t0+steps-1: out [steps][B][V] float32
__global__ void logits_kernel(SynthParams w, int t0, int steps, float* out) {
    const size_t total = (size_t)steps * w.B * w.V;
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
         i += (size_t)gridDim.x * blockDim.x) {
        const int v = (int)(i % w.V);
        const size_t r = i / w.V;
        const int b = (int)(r % w.B);
        const int t = t0 + (int)(r / w.B);
        float sigma = w.sigma;
        for (int k = 0; k < w.n_flat; ++k) if (w.flat[k] == t) sigma = w.flat_sigma;
        const float z = gauss(draw(key_of(w, KIND_LOGIT, 0, b), (uint64_t)t * w.V + v), w.ih_scale);
        out[i] = __fmul_rn(z, sigma);
    }
}

int grid_for(size_t total) {
    size_t blocks = (total + 255) / 256;
    return (int)(blocks < 65536 ? (blocks ? blocks : 1) : 65536);
}

}  // namespace

extern "C" {

int synth_kv_rows(const SynthParams* w, int layer, int seq, int64_t p0, int64_t n, void* K,
                  void* V, void* stream) {
    const size_t total = (size_t)n * w->Hkv * w->D;
    hipLaunchKernelGGL(kv_kernel, dim3(grid_for(total)), dim3(256), 0, (hipStream_t)stream, *w,
                       layer, seq, p0, n, K, V);
    return (int)hipGetLastError();
}

int synth_new_kv(const SynthParams* w, int t0, int steps, const int32_t* plen, void* K, void* V,
                 void* stream) {
    const size_t total = (size_t)steps * w->L * w->B * w->Hkv * w->D;
    hipLaunchKernelGGL(new_kv_kernel, dim3(grid_for(total)), dim3(256), 0, (hipStream_t)stream,
                       *w, t0, steps, plen, K, V);
    return (int)hipGetLastError();
}

int synth_q(const SynthParams* w, int t0, int steps, void* Q, void* stream) {
    const size_t total = (size_t)steps * w->L * w->B * w->Hq * w->D;
    hipLaunchKernelGGL(q_kernel, dim3(grid_for(total)), dim3(256), 0, (hipStream_t)stream, *w,
                       t0, steps, Q);
    return (int)hipGetLastError();
}

int synth_logits(const SynthParams* w, int t0, int steps, float* out, void* stream) {
    const size_t total = (size_t)steps * w->B * w->V;
    hipLaunchKernelGGL(logits_kernel, dim3(grid_for(total)), dim3(256), 0, (hipStream_t)stream,
                       *w, t0, steps, out);
    return (int)hipGetLastError();
}

}  // extern "C"
