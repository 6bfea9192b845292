"""MI355X-native beam-search decoder step (libmtstep) for a shallow attentional cGRU model."""
