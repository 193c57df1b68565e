"""Packed-storage accounting (test infrastructure only).

Paper section 4 ("Training"): storage is reported as the packed weight size
at the realised mean bit-width, so a model of P parameters at mean width
b_bar occupies P * b_bar / 8 bytes; FP16 stores 16 bits per weight.  Table 1
prints these sizes for the TinyStories ladder.  Per-group scales are not part
of that figure.
"""


def packed_bytes(params, mean_bits):
    """Bytes of packed codes for `params` weights at `mean_bits` bits each."""
    return params * mean_bits / 8.0


def fp16_bytes(params):
    return params * 2.0


def mean_bits(bit_counts):
    """Mean width of a population given {width: count}."""
    total = sum(bit_counts.values())
    return sum(b * n for b, n in bit_counts.items()) / total
