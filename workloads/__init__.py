"""Seeded synthetic workloads (shapes, weights, token batches). No method arithmetic."""
from .configs import Workload, WORKLOADS, get, PAD_ID, UNK_ID, BOS_ID, EOS_ID
from .gen import weight_specs, make_weights, make_batch, make_targets, round_bf16, WEIGHT_SEED
