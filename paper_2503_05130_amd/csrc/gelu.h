// GELU and its derivative for gfx950 device code.
//
// GELU(u) = u/2 (1 + erf(u / sqrt 2)) = u Phi(u), with erf from Abramowitz &
// Stegun, Handbook of Mathematical Functions, formula 7.1.26 (|error| <=
// 1.5e-7 for x >= 0): erfc(x) ~= (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5)
// exp(-x^2), t = 1 / (1 + p x).  Written through erfc so that u < 0 keeps its
// relative accuracy: Phi(u) = 1 - erfc(x)/2 for u >= 0 and erfc(x)/2 for
// u < 0, x = |u| / sqrt 2.  About 14 VALU operations instead of a full erff.
//
// GELU'(u) = Phi(u) + u phi(u), phi(u) = exp(-u^2 / 2) / sqrt(2 pi): the same
// exp(-x^2) serves both terms.
#pragma once

namespace iefwd {

struct GeluParts {
    float phi_cdf;   // Phi(u)
    float e;         // exp(-u^2 / 2)
};

__device__ inline GeluParts gelu_parts(float u) {
    const float x = fabsf(u) * 0.7071067811865476f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
    float poly = fmaf(1.061405429f, t, -1.453152027f);
    poly = fmaf(poly, t, 1.421413741f);
    poly = fmaf(poly, t, -0.284496736f);
    poly = fmaf(poly, t, 0.254829592f);
    const float e = __builtin_amdgcn_exp2f(-x * x * 1.4426950408889634f);
    const float erfc_x = poly * t * e;
    return {u >= 0.f ? fmaf(-0.5f, erfc_x, 1.0f) : 0.5f * erfc_x, e};
}

__device__ inline float gelu(float u) { return u * gelu_parts(u).phi_cdf; }

__device__ inline float gelu_grad(float u) {
    const GeluParts g = gelu_parts(u);
    return fmaf(u * 0.3989422804014327f, g.e, g.phi_cdf);
}

}  // namespace iefwd
