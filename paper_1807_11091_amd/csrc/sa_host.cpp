// Host-side helpers: error reporting and argument validation.  Every entry
// point validates all of its arguments here before anything is enqueued.
#include "sa_host.h"

#include <cstdio>
#include <cstring>

namespace sa {

static thread_local char g_err[512];

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_err[0] = '\0'; }

int check_hip(hipError_t e, const char *what) {
    if (e == hipSuccess) return SA_OK;
    return fail(SA_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

static const int64_t kMaxElems = (int64_t(1) << 31) - 1;

int validate_project(const sa_project_desc &d, int i) {
    if (d.A <= 0 || d.B <= 0 || d.C <= 0 || d.D <= 0)
        return fail(SA_E_ARG, "layer %d: shape [%lld,%lld,%lld,%lld] must be positive", i,
                    (long long)d.A, (long long)d.B, (long long)d.C, (long long)d.D);
    if (d.A > kMaxElems / d.B || d.A * d.B > kMaxElems / (d.C * d.D) || d.C * d.D > kMaxElems)
        return fail(SA_E_ARG, "layer %d: A*B*C*D must be below 2^31", i);
    if (d.groups <= 0 || d.A % d.groups != 0)
        return fail(SA_E_ARG, "layer %d: groups=%d must be >= 1 and divide A=%lld", i, d.groups,
                    (long long)d.A);
    if (d.kind < SA_FILTER || d.kind > SA_ELEMENT)
        return fail(SA_E_ARG, "layer %d: unknown kind %d", i, d.kind);
    int64_t G = n_groups(d);
    if (d.k < 0 || d.k > G)
        return fail(SA_E_ARG, "layer %d: k=%lld outside [0, n_groups=%lld]", i, (long long)d.k,
                    (long long)G);
    if (d.kind != SA_ELEMENT && G > SA_MAX_STRUCT_GROUPS)
        return fail(SA_E_UNSUPPORTED, "layer %d: %lld groups exceed the structured selection limit %d",
                    i, (long long)G, SA_MAX_STRUCT_GROUPS);
    if (!d.W || !d.U || !d.Z || !d.mask || (d.k > 0 && !d.kept_idx))
        return fail(SA_E_ARG, "layer %d: W, U, Z, mask and (for k > 0) kept_idx are required", i);
    if (!aligned(d.W, 16) || !aligned(d.U, 16) || !aligned(d.Z, 16) || (d.G && !aligned(d.G, 16)))
        return fail(SA_E_ALIGN, "layer %d: W, U, Z and G must be 16-byte aligned", i);
    if (d.scores && !aligned(d.scores, 8))
        return fail(SA_E_ALIGN, "layer %d: scores must be 8-byte aligned", i);
    if (d.kept_idx && !aligned(d.kept_idx, 4))
        return fail(SA_E_ALIGN, "layer %d: kept_idx must be 4-byte aligned", i);
    if ((const void *)d.Z == (const void *)d.W || d.Z == d.U)
        return fail(SA_E_ARG, "layer %d: Z must not alias W or U", i);
    if (d.G && ((const void *)d.G == (const void *)d.W || d.G == d.U || d.G == d.Z))
        return fail(SA_E_ARG, "layer %d: G must not alias W, U or Z", i);
    return SA_OK;
}

int validate_dual(const sa_dual_desc &d, int i) {
    if (d.n <= 0 || d.n > kMaxElems)
        return fail(SA_E_ARG, "layer %d: n=%lld must be in [1, 2^31)", i, (long long)d.n);
    if (!d.W || !d.Z || !d.U)
        return fail(SA_E_ARG, "layer %d: W, Z and U are required", i);
    if (!d.update_dual && !d.G)
        return fail(SA_E_ARG, "layer %d: nothing to do (update_dual=0 and G=NULL)", i);
    if (!aligned(d.W, 16) || !aligned(d.Z, 16) || !aligned(d.U, 16) || (d.G && !aligned(d.G, 16)))
        return fail(SA_E_ALIGN, "layer %d: W, Z, U and G must be 16-byte aligned", i);
    return SA_OK;
}

int validate_sgd(const sa_sgd_desc &d, int i) {
    if (d.A <= 0 || d.B <= 0 || d.C <= 0 || d.D <= 0)
        return fail(SA_E_ARG, "layer %d: shape must be positive", i);
    if (d.A > kMaxElems / d.B || d.A * d.B > kMaxElems / (d.C * d.D))
        return fail(SA_E_ARG, "layer %d: A*B*C*D must be below 2^31", i);
    if (d.kind < SA_FILTER || d.kind > SA_ELEMENT) return fail(SA_E_ARG, "layer %d: unknown kind %d", i, d.kind);
    if (!d.W || !d.Gf) return fail(SA_E_ARG, "layer %d: W and Gf are required", i);
    if ((d.Z == nullptr) != (d.U == nullptr)) return fail(SA_E_ARG, "layer %d: give both Z and U or neither", i);
    if (d.Gf == d.W) return fail(SA_E_ARG, "layer %d: Gf must not alias W", i);
    if (!aligned(d.W, 16) || !aligned(d.Gf, 16) || (d.Z && (!aligned(d.Z, 16) || !aligned(d.U, 16))))
        return fail(SA_E_ALIGN, "layer %d: W, Gf, Z and U must be 16-byte aligned", i);
    return SA_OK;
}

int validate_compact(const sa_compact_desc &d) {
    if (d.A <= 0 || d.B <= 0 || d.C <= 0 || d.D <= 0)
        return fail(SA_E_ARG, "compact: shape must be positive");
    if (d.A > kMaxElems / d.B || d.A * d.B > kMaxElems / (d.C * d.D))
        return fail(SA_E_ARG, "compact: A*B*C*D must be below 2^31");
    if (d.groups <= 0 || d.groups > SA_MAX_CONV_GROUPS || d.A % d.groups != 0)
        return fail(SA_E_ARG, "compact: groups=%d must be in [1, %d] and divide A", d.groups,
                    SA_MAX_CONV_GROUPS);
    if (d.C > 255 || d.D > 255)
        return fail(SA_E_UNSUPPORTED, "compact: kernel %lldx%lld larger than 255", (long long)d.C,
                    (long long)d.D);
    if ((int64_t)d.groups * d.B > 32768)
        return fail(SA_E_UNSUPPORTED, "compact: more than 32768 input channels");
    if (!d.Z || !d.Wc || !d.row_idx || !d.col_ch || !d.col_tap || !d.ws)
        return fail(SA_E_ARG, "compact: Z, Wc, row_idx, col_ch, col_tap and ws are required");
    if (d.in_compacted && !d.in_ch_mask)
        return fail(SA_E_ARG, "compact: in_compacted requires in_ch_mask");
    if (!aligned(d.Wc, 16) || !aligned(d.ws, 256) || !aligned(d.row_idx, 4) ||
        !aligned(d.col_ch, 4) || !aligned(d.col_tap, 4) || !aligned(d.Z, 4))
        return fail(SA_E_ALIGN, "compact: Wc must be 16-byte, ws 256-byte, tables 4-byte aligned");
    return SA_OK;
}

int validate_conv(const sa_conv_desc &d) {
    if (!d.sizes)
        return fail(SA_E_ARG, "conv: sizes (from structadmm_compact) is required");
    const sa_compact_sizes &s = *d.sizes;
    if (d.N <= 0 || d.H <= 0 || d.W <= 0 || d.Cx <= 0 || d.C <= 0 || d.D <= 0 || d.stride <= 0 ||
        d.pad < 0)
        return fail(SA_E_ARG, "conv: N, H, W, Cx, C, D, stride must be positive and pad >= 0");
    if (s.groups <= 0 || s.groups > SA_MAX_CONV_GROUPS)
        return fail(SA_E_ARG, "conv: sizes->groups=%d out of range", s.groups);
    int64_t P = ((int64_t)d.H + 2 * d.pad - d.C) / d.stride + 1;
    int64_t Q = ((int64_t)d.W + 2 * d.pad - d.D) / d.stride + 1;
    if (d.H + 2 * d.pad < d.C || d.W + 2 * d.pad < d.D || P <= 0 || Q <= 0)
        return fail(SA_E_ARG, "conv: output would be empty");
    if ((int64_t)d.N * P * Q > kMaxElems || (int64_t)d.N * d.H * d.W > kMaxElems)
        return fail(SA_E_UNSUPPORTED, "conv: N*P*Q and N*H*W must be below 2^31");
    if ((int64_t)d.N * d.H * d.W * d.Cx >= (int64_t(1) << 40))
        return fail(SA_E_UNSUPPORTED, "conv: input too large");
    if (d.C > 255 || d.D > 255)
        return fail(SA_E_UNSUPPORTED, "conv: kernel larger than 255");
    int64_t Cy = 0;
    for (int g = 0; g < s.groups; ++g) {
        if (s.M[g] < 0 || s.K[g] < 0)
            return fail(SA_E_ARG, "conv: negative group size");
        if (s.K[g] > 16384)
            return fail(SA_E_UNSUPPORTED, "conv: K=%d columns exceed 16384", s.K[g]);
        if (s.run[g] > 0 && (int64_t)s.run[g] * d.C * d.D != s.K[g])
            return fail(SA_E_ARG, "conv: run[%d]=%d inconsistent with K=%d", g, s.run[g], s.K[g]);
        if (s.run[g] > 0 && s.run_base[g] + s.run[g] > d.Cx)
            return fail(SA_E_ARG, "conv: channel run of group %d exceeds Cx=%d", g, d.Cx);
        Cy += s.M[g];
    }
    if (Cy <= 0)
        return fail(SA_E_ARG, "conv: no output channels");
    if (d.ldy != 0 && d.ldy < Cy)
        return fail(SA_E_ARG, "conv: ldy=%d is below the %lld output channels", d.ldy, (long long)Cy);
    if (!d.X || !d.Wc || !d.Y || !d.col_ch || !d.col_tap)
        return fail(SA_E_ARG, "conv: X, Wc, col_ch, col_tap and Y are required");
    if (!aligned(d.X, 16) || !aligned(d.Wc, 16) || !aligned(d.Y, 4))
        return fail(SA_E_ALIGN, "conv: X and Wc must be 16-byte aligned, Y 4-byte aligned");
    return SA_OK;
}

}  // namespace sa

extern "C" const char *structadmm_last_error(void) { return sa::g_err; }

extern "C" const char *structadmm_version(void) { return "structadmm-gfx950 0.1"; }
