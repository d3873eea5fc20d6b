"""Offline training of the format predictor (the paper's Sec. 4.3-4.5).

``collect`` profiles every feasible format of each training matrix on the GPU
through the library's exhaustive selector (GS_SEL_PROFILE) and records the
features; ``train`` fits a boosted tree ensemble on the min-max normalised
features and writes it in the library's model format (``model.gsm``), which
``SelectContext("model")`` loads by default.
"""
import os

MODEL_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "model.gsm")
DATA_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "data.csv")
