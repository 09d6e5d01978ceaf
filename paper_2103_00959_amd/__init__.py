"""MI355X-native GNN message-passing operators (CogDL, arxiv 2103.00959, section 2.2)."""
