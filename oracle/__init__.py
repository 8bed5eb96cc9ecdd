"""CPU oracle for XPipe's one-stage training step (fp64 numpy).

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow reference that the
GPU path is checked against.  It shares no code with the GPU library and
never imports it.  Only tests/, __graft_entry__.smoke() and the cpu_baseline
leg of bench.py may import or run anything here; the product path must never
route through it.

Contents:
  method  Eq. 1 / Eq. 2 version difference, Eq. 3 / Eq. 4 prediction, Adam update,
          momentum-SGD and RMSProp updates that keep the prediction's Adam moments
  layers  layer forwards and VJPs (conv, linear, BN, ReLU, pools, GAP, CE)
  stage   a stage's forward, backward-with-recompute, the mini-batch driver and
          the driver of one GPU's part of the interleaved schedule
  schedule  the pipeline schedule as a unit-time model, with staleness counts
"""
from .method import (HALF_DOWN, HALF_EVEN, HALF_UP, PRED_ADAMDIR, PRED_EQ3, PRED_LITERAL,
                     PRED_SMOOTHED,
                     RULE_ADAM, RULE_MOMENTUM_SGD, RULE_RMSPROP, adam_moments, adam_update,
                     momentum_sgd_update, predict, rmsprop_update, version_difference_bwd,
                     version_difference_fwd)
from .stage import Hyper, MinibatchRecord, ScheduleRecord, Stage, train_schedule, train_stage
from . import schedule

__all__ = [
    "HALF_DOWN", "HALF_EVEN", "HALF_UP", "PRED_ADAMDIR", "PRED_EQ3", "PRED_LITERAL", "PRED_SMOOTHED",
    "RULE_ADAM", "RULE_MOMENTUM_SGD", "RULE_RMSPROP", "adam_moments", "adam_update",
    "momentum_sgd_update", "predict", "rmsprop_update", "version_difference_bwd",
    "version_difference_fwd",
    "Hyper", "MinibatchRecord", "ScheduleRecord", "Stage", "train_schedule", "train_stage",
    "schedule",
]
