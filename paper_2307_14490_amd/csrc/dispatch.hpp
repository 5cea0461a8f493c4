// Instantiation over the supported row shapes: G lanes per row (power of two,
// 1..64) and C float4 chunks per lane (C > 1 only with G = 64), D <= 1024.
#pragma once

#define HUGE_ROW_CASE(GG, CC, ...)           \
    case (GG) * 8 + (CC): {                  \
        constexpr int G_ = (GG);             \
        constexpr int C_ = (CC);             \
        __VA_ARGS__;                         \
    } break;

#define HUGE_ROW_DISPATCH(rs, ...)                   \
    switch ((rs).G * 8 + (rs).C) {                   \
        HUGE_ROW_CASE(1, 1, __VA_ARGS__)             \
        HUGE_ROW_CASE(2, 1, __VA_ARGS__)             \
        HUGE_ROW_CASE(4, 1, __VA_ARGS__)             \
        HUGE_ROW_CASE(8, 1, __VA_ARGS__)             \
        HUGE_ROW_CASE(16, 1, __VA_ARGS__)            \
        HUGE_ROW_CASE(32, 1, __VA_ARGS__)            \
        HUGE_ROW_CASE(64, 1, __VA_ARGS__)            \
        HUGE_ROW_CASE(64, 2, __VA_ARGS__)            \
        HUGE_ROW_CASE(64, 3, __VA_ARGS__)            \
        HUGE_ROW_CASE(64, 4, __VA_ARGS__)            \
        default:                                     \
            return hipErrorInvalidValue;             \
    }

// Negative rows in flight in the step kernels: the smallest supported block
// that holds min(K, 8) rows.
inline int neg_block(int K) {
    const int want = K < 8 ? K : 8;
    const int blocks[] = {2, 3, 4, 5, 6, 8};
    for (int b : blocks)
        if (b >= want) return b;
    return 8;
}

#define HUGE_NEG_CASE(NN, ...)        \
    case (NN): {                      \
        constexpr int NB_ = (NN);     \
        __VA_ARGS__;                  \
    } break;

#define HUGE_NEG_DISPATCH(nb, ...)           \
    switch (nb) {                            \
        HUGE_NEG_CASE(2, __VA_ARGS__)        \
        HUGE_NEG_CASE(3, __VA_ARGS__)        \
        HUGE_NEG_CASE(4, __VA_ARGS__)        \
        HUGE_NEG_CASE(5, __VA_ARGS__)        \
        HUGE_NEG_CASE(6, __VA_ARGS__)        \
        HUGE_NEG_CASE(8, __VA_ARGS__)        \
        default:                             \
            return hipErrorInvalidValue;     \
    }

// Whether the negatives form one block of the block size (K == NB): F_.
#define HUGE_FULL_DISPATCH(full, ...)      \
    if (full) {                            \
        constexpr bool F_ = true;          \
        __VA_ARGS__;                       \
    } else {                               \
        constexpr bool F_ = false;         \
        __VA_ARGS__;                       \
    }

// Element type of the tables: E_ is float or bf16_t.
#define HUGE_ELEM_DISPATCH(dtype, ...)      \
    if ((dtype) == kDtypeBf16) {            \
        using E_ = bf16_t;                  \
        __VA_ARGS__;                        \
    } else {                                \
        using E_ = float;                   \
        __VA_ARGS__;                        \
    }

// Unit layouts of bf16 rows (8 elements per unit), D <= 1024: G lanes per
// row and U units per lane.
#define HUGE_PAIR_CASE(GG, UU, ...)          \
    case (GG) * 8 + (UU): {                  \
        constexpr int G_ = (GG);             \
        constexpr int U_ = (UU);             \
        __VA_ARGS__;                         \
    } break;

#define HUGE_PAIR_DISPATCH(ps, ...)                  \
    switch ((ps).G * 8 + (ps).U) {                   \
        HUGE_PAIR_CASE(1, 1, __VA_ARGS__)            \
        HUGE_PAIR_CASE(2, 1, __VA_ARGS__)            \
        HUGE_PAIR_CASE(4, 1, __VA_ARGS__)            \
        HUGE_PAIR_CASE(8, 1, __VA_ARGS__)            \
        HUGE_PAIR_CASE(16, 1, __VA_ARGS__)           \
        HUGE_PAIR_CASE(32, 1, __VA_ARGS__)           \
        HUGE_PAIR_CASE(64, 1, __VA_ARGS__)           \
        HUGE_PAIR_CASE(64, 2, __VA_ARGS__)           \
        default:                                     \
            return hipErrorInvalidValue;             \
    }
