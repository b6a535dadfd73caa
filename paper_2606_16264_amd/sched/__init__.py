"""Host-side scheduling layer above the layer step: an iteration-latency
predictor fitted to measured steps, and the SLO slack accounting and
discrete-event simulator of prefill/decode multiplexing built on it."""
from .predictor import LatencyModel, batch_features, FEATURES  # noqa: F401
