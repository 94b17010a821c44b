"""The five synthetic translation workloads, by name.

Each entry fixes the model shape (Section 2 "Background" and Section 4.3 of the
OpenNMT paper name the pieces: stacked LSTM encoder, optionally bidirectional,
input-feeding LSTM decoder, global "general" attention, softmax generator) and
the search/batch shape (Table 2: 2x500 RNN, batch 64, beam 5; Section 5:
default length filter of 50 tokens; Table 3: bi-RNN, max length 100).

Nothing here computes anything of the method; it is plain data.
"""

from dataclasses import dataclass, asdict

PAD_ID, UNK_ID, BOS_ID, EOS_ID = 0, 1, 2, 3


@dataclass(frozen=True)
class Workload:
    name: str
    index: int            # 1-based position in the list below (data seed = 1000 + index)
    enc_layers: int
    dec_layers: int
    bidirectional: bool
    emb: int
    hidden: int           # decoder hidden size H; the encoder uses H/2 per direction when bidirectional
    src_vocab: int
    tgt_vocab: int
    batch: int
    len_lo: int
    len_hi: int           # source lengths uniform in [len_lo, len_hi], padded to len_hi
    beam: int
    max_len: int          # at most this many generated tokens, EOS included
    alpha: float          # GNMT length-normalisation exponent
    wdtype: str           # "fp32" or "bf16" (weights rounded to bfloat16, fp32 accumulation)
    zipf_s: float         # exponent of the bounded Zipf source-token distribution
    attn: str = "general"  # attention score: "general" q.W_a m, "dot" q.m, "concat" v_a.tanh(W_a [q; m])

    @property
    def enc_hidden(self) -> int:
        return self.hidden // 2 if self.bidirectional else self.hidden

    @property
    def s_max(self) -> int:
        return self.len_hi

    def as_dict(self):
        return asdict(self)


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny", 1, 1, 1, False, 32, 64, 1000, 1000, 4, 6, 10, 2, 12, 0.0, "fp32", 1.0),
        Workload("default", 2, 2, 2, False, 500, 500, 50000, 50000, 64, 10, 50, 5, 100, 0.0, "fp32", 1.0),
        Workload("larger", 3, 4, 4, True, 1000, 1000, 50000, 50000, 64, 10, 60, 5, 120, 0.0, "bf16", 1.0),
        Workload("greedy", 4, 2, 2, False, 512, 1024, 32000, 32000, 512, 15, 40, 1, 80, 0.0, "bf16", 1.1),
        Workload("long", 5, 2, 2, False, 500, 500, 50000, 50000, 16, 150, 200, 10, 250, 0.6, "fp32", 1.0),
    ]
}

BY_INDEX = {w.index: w for w in WORKLOADS.values()}


def get(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return BY_INDEX[name_or_index]
    return WORKLOADS[name_or_index]
